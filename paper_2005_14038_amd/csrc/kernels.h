// Internal launch interface of the gfx950 kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace hp {

// Geometry of one convolution (FC layers are 1x1 convolutions on a 1x1 map).
struct ConvGeo {
    int N, H, W, C;   // input  [N][H][W][C]
    int K, R, S;      // weight [K][R][S][C]
    int P, Q;         // output [N][P][Q][K]
    int st, pad;
};

enum GemmOp { OP_FWD = 0, OP_DGRAD = 1, OP_WGRAD = 2 };

// Implicit-GEMM contraction on MFMA.
//   OP_FWD:   out[N*P*Q][K]   = conv(x, w) (+ bias) (relu)
//   OP_DGRAD: out[N*H*W][C]   = dgrad(dy, w)        (accumulate adds into out)
//   OP_WGRAD: out[K][R*S*C]   = wgrad(x, dy)
// `a` is x (FWD, WGRAD) or dy (DGRAD); `b` is w (FWD, DGRAD) or dy (WGRAD).
struct GemmPlan {
    int op;
    int bf16;          // round operands to bf16 (RNE) when staging
    int h16;           // bf16: the geometry allows bf16 operands in memory (launch_gemm a16/b16)
    int h16k;          // h16 and both operands k-major (FWD; DGRAD with stride 1 or 2 and b16t)
    int h16d;          // h16k on the 256 x 128 direct-to-LDS kernel (FWD, stride-1 DGRAD)
    int wide;          // fp32 with the wide (LDS-staged, 16-byte) epilogue: short reductions
    int fcf;           // fp32 forward of a fully connected layer on fcf_kernel
    int fcw;           // fp32 weight gradient of a fully connected layer on fcw_kernel
    int bias_col;      // OP_WGRAD: Ncols includes the bias-gradient column
    int cfg;           // tile configuration
    int tfull;         // tiles computed whole (one workgroup each)
    int splits;        // the other tiles are cut into `splits` reduction chunks
    int kchunk;        // reduction length of a chunk (multiple of the K tile)
    int nwg;           // workgroups launched
    int bm, bn;        // workgroup tile
    size_t ws_floats;  // workspace for the partial tiles of the cut tiles
    long M, Ncols, Kred;
};

// bias_col (OP_WGRAD only): append a column of ones to the gathered input so
// that the last output column is sum_m dy[m][k], the bias gradient.  The plan
// keeps it only when it costs no extra tile; plan.bias_col says whether it did.
// allow_h16d = 0 keeps the plan off the 256 x 128 direct-to-LDS kernel (whose
// epilogue writes no column statistics).
GemmPlan plan_gemm(int op, const ConvGeo& g, int bf16, int num_cus, int bias_col = 0,
                   int allow_h16d = 1);

// epilogue flags
enum {
    EPI_BIAS = 1,     // out += bias[col]
    EPI_RELU = 2,     // out = max(out, 0)
    EPI_ACCUM = 4,    // out += previous out
    EPI_MASK = 8,     // out = mask[row][col] > 0 ? out : 0   (ReLU backward fused)
    EPI_BIASCOL = 16  // last column (see plan_gemm bias_col) goes to bias_out[row]
};

struct Epilogue {
    int flags = 0;
    const float* bias = nullptr;
    const float* mask = nullptr;
    float* bias_out = nullptr;
    // optional (flags within EPI_BIAS): per output column and row tile of
    // plan.bm rows, the tile's mean and sum of squared deviations from it:
    // stats[t * Ncols + col] and stats[(tiles_m + t) * Ncols + col]
    float* stats = nullptr;
    // optional (not with stats or a bias-gradient column; 16-byte aligned):
    // each final output element also written rounded to bf16 (nearest even)
    uint16_t* out16 = nullptr;
};

// a16 / b16 (bf16 plans with plan.h16, optional): the same operands already
// rounded to bf16, 16-byte aligned; when given, the kernel stages them directly.
// b16t (OP_DGRAD, optional): the weights transposed to [C][R][S][K] in bf16;
// with it a plan with h16k runs on k-major operands.
// Whether launch_gemm writes Epilogue::stats for this plan and epilogue flags.
bool plan_stats(const GemmPlan& plan, int flags);
hipError_t launch_gemm(const GemmPlan& plan, const ConvGeo& g, const float* a,
                       const float* b, float* out, const Epilogue& ep, float* ws,
                       hipStream_t s, const uint16_t* a16 = nullptr,
                       const uint16_t* b16 = nullptr, const uint16_t* b16t = nullptr);

// dst[i] = bf16(src[i]) (round to nearest even), n elements
hipError_t launch_cast_bf16(const float* src, uint16_t* dst, size_t n, hipStream_t s);

// Channel padding: dst[r][c] = src[r][c] (c < C), 0 (C <= c < Cp), rows x Cp,
// into dst (fp32) or, when dst16 is given, dst16 (bf16, nearest even).
hipError_t launch_pad_channels(const float* src, float* dst, uint16_t* dst16, size_t rows, int C,
                               int Cp, hipStream_t s);
// The reverse: dst[r][c] = src[r][c] for c < C (src rows of Cp).
hipError_t launch_unpad_channels(const float* src, float* dst, size_t rows, int C, int Cp,
                                 hipStream_t s);

// Transposed bf16 weight copies for the data gradient on k-major operands:
// for each table layer, dst[off + (c*RS + rs)*K + k] = bf16(src[off + (k*RS + rs)*C + c]).
// tile0 = the layer's first WT_TILE x WT_TILE tile number (prefix sums of wt_tiles, in
// table order); `tiles` = the total.  The table lives in device memory.
struct WtLayer {
    long off;
    int K, RS, C, tile0;
};
constexpr int WT_TILE = 64;
inline int wt_tiles(int K, int RS, int C) {
    return RS * ((K + WT_TILE - 1) / WT_TILE) * ((C + WT_TILE - 1) / WT_TILE);
}
hipError_t launch_cast_bf16_t(const float* src, uint16_t* dst, const WtLayer* table,
                              int nlayers, int tiles, hipStream_t s);

// ---- element-wise / reduction kernels (elementwise.hip) -------------------
// y = max(x, 0)
hipError_t launch_relu_fwd(const float* x, float* y, size_t n, hipStream_t s);
// dx = dy * (y > 0); with accumulate, dx += ...
hipError_t launch_relu_bwd(const float* y, const float* dy, float* dx, size_t n,
                           int accumulate, hipStream_t s);
// out = a + b (relu optional)
// y16 (optional): also write y rounded to bf16
hipError_t launch_add_fwd(const float* a, const float* b, float* y, size_t n, int relu,
                          hipStream_t s, uint16_t* y16 = nullptr);
// out = v (accumulate = 0) or out += v
hipError_t launch_copy_or_acc(const float* v, float* out, size_t n, int accumulate,
                              hipStream_t s);
// arg (optional, one byte per output element, R * S < 256): records the
// window tap of every first maximum for the backward pass
hipError_t launch_maxpool_fwd(const float* x, float* y, int N, int H, int W, int C, int R,
                              int S, int st, int pad, int P, int Q, hipStream_t s,
                              uint16_t* y16 = nullptr, uint8_t* arg = nullptr);
// windows that tile the input exactly (the backward needs no recorded taps)
bool maxpool_tiled(int H, int W, int R, int S, int st, int pad, int P, int Q);
// mask (optional, layout of dx): the pooled input is a ReLU output; dx is
// zeroed where mask <= 0 (ReLU backward fused).  arg (optional): the taps the
// forward pass recorded, used for overlapping windows instead of recomputing
// each window's maximum from x.
// dx16 (optional): also write the final dx rounded to bf16 (nearest even)
hipError_t launch_maxpool_bwd(const float* x, const float* dy, float* dx, int N, int H, int W,
                              int C, int R, int S, int st, int pad, int P, int Q,
                              int accumulate, const float* mask, hipStream_t s,
                              const uint8_t* arg = nullptr, uint16_t* dx16 = nullptr);
hipError_t launch_gap_fwd(const float* x, float* y, int N, int HW, int C, hipStream_t s);
hipError_t launch_gap_bwd(const float* dy, float* dx, int N, int HW, int C, int accumulate,
                          hipStream_t s);

// Per-channel column reductions over M rows of an [M][C] matrix, deterministic:
// partial sums over row blocks, then a fixed-order finalisation.
size_t colsum_ws_floats(long M, int C);
// out[c] = sum_m v[m][c]  (out may be a device pointer into a gradient vector)
hipError_t launch_colsum(const float* v, long M, int C, float* out, float* ws, hipStream_t s);

// Batch-norm (training mode).  Statistics: mean[c], invstd[c] = 1/sqrt(var+eps)
// with the biased variance; apply: y = gamma*(x-mean)*invstd + beta (relu opt.).
size_t bn_ws_floats(long M, int C);
hipError_t launch_bn_fwd(const float* x, long M, int C, const float* gamma, const float* beta,
                         float eps, float* y, float* mean, float* invstd, int relu, float* ws,
                         hipStream_t s, uint16_t* y16 = nullptr);
// The same from per-row-block partials computed elsewhere (the producing
// contraction's tile statistics): part0[b][c] = mean of block b, part1[b][c]
// = its sum of squared deviations, blocks of rb rows (the last one shorter).
hipError_t launch_bn_fwd_partials(const float* x, long M, int C, const float* gamma,
                                  const float* beta, float eps, float* y, float* mean,
                                  float* invstd, int relu, const float* part0, const float* part1,
                                  int nb, long rb, hipStream_t s, uint16_t* y16 = nullptr);
// Backward.  If relu_y != NULL the incoming gradient is first masked by
// relu_y > 0 (BN followed by ReLU).  Writes dgamma, dbeta and, unless dx is NULL,
// dx (accumulate optional).
hipError_t launch_bn_bwd(const float* x, const float* dy, const float* relu_y, long M, int C,
                         const float* gamma, const float* mean, const float* invstd, float* dx,
                         float* dgamma, float* dbeta, int accumulate, float* ws, hipStream_t s,
                         uint16_t* dx16 = nullptr);

// Softmax cross-entropy: loss (one float) = mean_n (lse(z_n) - z_n[label]);
// dz = (softmax(z) - onehot) / B.
hipError_t launch_softmax_ce(const float* z, const int32_t* labels, int B, int K, float* loss,
                             float* dz, float* ws, hipStream_t s);


// ---- WSP kernels (wsp.hip) ------------------------------------------------
// u = (-lr)*g; dst = newest + u; ut = first ? u : ut + u   (no FMA contraction)
hipError_t launch_wsp_local_update(const float* g, const float* newest, float* dst, float* ut,
                                   size_t n, float lr, int first, hipStream_t s);
// with momentum: v = mu*v + g; u = (-lr)*v; then as above
hipError_t launch_wsp_local_update_momentum(const float* g, const float* newest, float* dst,
                                            float* ut, float* vel, size_t n, float lr, float mu,
                                            int first, hipStream_t s);
// wg = wg + ut
hipError_t launch_wsp_push(float* wg, const float* ut, size_t n, hipStream_t s);
// dst = src
hipError_t launch_wsp_copy(const float* src, float* dst, size_t n, hipStream_t s);
// wave end fused: the local update (momentum when vel != nullptr), then
// w_g = w_g + u~, then dst = w_g (pull != 0) or dst = newest + u
hipError_t launch_wsp_wave_end(const float* g, const float* newest, float* dst, float* ut,
                               float* vel, float* wg, size_t n, float lr, float mu, int first,
                               int pull, hipStream_t s);

}  // namespace hp
