// Element-wise and per-channel reduction kernels of the stage step (gfx950):
// ReLU, residual add, max-pool, global average pool, batch-norm, softmax
// cross-entropy and column sums (bias gradients).
//
// Layout is NHWC throughout, so a "channel" is the fastest axis: consecutive
// lanes of a wave64 walk consecutive channels and every global access is
// coalesced.  Per-channel reductions over the M = N*H*W rows are done in two
// deterministic passes: each workgroup reduces a fixed block of rows for a
// strip of channels into a partial row of a workspace, then one thread per
// channel adds the partials in block order.  No atomics are used, so every
// result is bit-reproducible run to run.
#include "kernels.h"

namespace hp {
namespace {

constexpr int EW_THREADS = 256;

inline int ew_blocks(size_t n) {
    size_t b = (n + EW_THREADS - 1) / EW_THREADS;
    return (int)(b < 16384 ? (b ? b : 1) : 16384);
}

__global__ void relu_fwd_kernel(const float* __restrict__ x, float* __restrict__ y, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        y[i] = fmaxf(x[i], 0.f);
}

__global__ void relu_bwd_kernel(const float* __restrict__ y, const float* __restrict__ dy,
                                float* __restrict__ dx, size_t n, int acc) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        float v = y[i] > 0.f ? dy[i] : 0.f;
        dx[i] = acc ? dx[i] + v : v;
    }
}

__global__ void add_fwd_kernel(const float* __restrict__ a, const float* __restrict__ b,
                               float* __restrict__ y, size_t n, int relu) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        float v = a[i] + b[i];
        y[i] = relu ? fmaxf(v, 0.f) : v;
    }
}

__global__ void copy_or_acc_kernel(const float* __restrict__ v, float* __restrict__ out, size_t n,
                                   int acc) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        out[i] = acc ? out[i] + v[i] : v[i];
}

// max-pool forward: padded taps never win; the first maximum in row-major
// window order is kept (strict '>' comparison).
__global__ void maxpool_fwd_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int H,
                                   int W, int C, int R, int S, int st, int pad, int P, int Q) {
    const size_t total = (size_t)N * P * Q * C;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        size_t t = i / C;
        int q = (int)(t % Q); t /= Q;
        int p = (int)(t % P);
        int n = (int)(t / P);
        float m = -INFINITY;
        bool any = false;
        for (int r = 0; r < R; ++r) {
            int h = p * st - pad + r;
            if (h < 0 || h >= H) continue;
            for (int s = 0; s < S; ++s) {
                int w = q * st - pad + s;
                if (w < 0 || w >= W) continue;
                float v = x[(((size_t)n * H + h) * W + w) * C + c];
                if (!any || v > m) { m = v; any = true; }
            }
        }
        y[i] = m;
    }
}

// max-pool backward as a gather: each input element sums dy over the windows
// whose first maximum it is (the window's argmax is recomputed from x).
__global__ void maxpool_bwd_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                   float* __restrict__ dx, int N, int H, int W, int C, int R,
                                   int S, int st, int pad, int P, int Q, int acc,
                                   const float* __restrict__ mask) {
    const size_t total = (size_t)N * H * W * C;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        size_t t = i / C;
        int w0 = (int)(t % W); t /= W;
        int h0 = (int)(t % H);
        int n = (int)(t / H);
        float sum = 0.f;
        for (int r = 0; r < R; ++r) {
            int tp = h0 + pad - r;
            if (tp < 0 || tp % st) continue;
            int p = tp / st;
            if (p >= P) continue;
            for (int s = 0; s < S; ++s) {
                int tq = w0 + pad - s;
                if (tq < 0 || tq % st) continue;
                int q = tq / st;
                if (q >= Q) continue;
                // first argmax of window (p, q)
                int best = -1;
                float m = -INFINITY;
                for (int rr = 0; rr < R; ++rr) {
                    int h = p * st - pad + rr;
                    if (h < 0 || h >= H) continue;
                    for (int ss = 0; ss < S; ++ss) {
                        int w = q * st - pad + ss;
                        if (w < 0 || w >= W) continue;
                        float v = x[(((size_t)n * H + h) * W + w) * C + c];
                        if (best < 0 || v > m) { m = v; best = rr * S + ss; }
                    }
                }
                if (best == r * S + s) sum += dy[(((size_t)n * P + p) * Q + q) * C + c];
            }
        }
        if (mask && !(mask[i] > 0.f)) sum = 0.f;
        dx[i] = acc ? dx[i] + sum : sum;
    }
}

// max-pool backward for non-overlapping windows (window = stride, no padding,
// windows tile the input exactly): one thread per output element writes its
// whole window -- dy at the first maximum, zero elsewhere.
template <int RT>   // RT > 0: window size fixed at compile time; 0: runtime R
__global__ void maxpool_bwd_tiled_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                         float* __restrict__ dx, int N, int H, int W, int C, int Rr,
                                         int P, int Q, int acc, const float* __restrict__ mask) {
    const int R = RT > 0 ? RT : Rr;
    const size_t total = (size_t)N * P * Q * C;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        size_t t = i / C;
        int q = (int)(t % Q); t /= Q;
        int p = (int)(t % P);
        int n = (int)(t / P);
        const size_t base = (((size_t)n * H + p * R) * W + q * R) * C + c;
        const float g = dy[i];
        if constexpr (RT > 0) {
            // taps kept in registers; when pooling a ReLU output the taps are the mask
            float v[RT * RT];
            int best = 0;
#pragma unroll
            for (int k = 0; k < RT * RT; ++k) {
                v[k] = x[base + ((size_t)(k / RT) * W + k % RT) * C];
                if (v[k] > v[best]) best = k;
            }
#pragma unroll
            for (int k = 0; k < RT * RT; ++k) {
                size_t j = base + ((size_t)(k / RT) * W + k % RT) * C;
                float o = (k == best) ? g : 0.f;
                if (mask && !((mask == x ? v[k] : mask[j]) > 0.f)) o = 0.f;
                dx[j] = acc ? dx[j] + o : o;
            }
        } else {
            int best = 0;
            float m = x[base];
            for (int r = 0; r < R; ++r)
                for (int s = 0; s < R; ++s) {
                    float v = x[base + ((size_t)r * W + s) * C];
                    if (v > m) { m = v; best = r * R + s; }
                }
            for (int r = 0; r < R; ++r)
                for (int s = 0; s < R; ++s) {
                    size_t j = base + ((size_t)r * W + s) * C;
                    float o = (r * R + s == best) ? g : 0.f;
                    if (mask && !(mask[j] > 0.f)) o = 0.f;
                    dx[j] = acc ? dx[j] + o : o;
                }
        }
    }
}

__global__ void gap_fwd_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int HW,
                               int C) {
    const size_t total = (size_t)N * C;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        int n = (int)(i / C);
        float s = 0.f;
        for (int j = 0; j < HW; ++j) s += x[((size_t)n * HW + j) * C + c];
        y[i] = s / (float)HW;
    }
}

__global__ void gap_bwd_kernel(const float* __restrict__ dy, float* __restrict__ dx, int N, int HW,
                               int C, int acc) {
    const size_t total = (size_t)N * HW * C;
    const float inv = 1.f / (float)HW;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        int n = (int)(i / ((size_t)HW * C));
        float v = dy[(size_t)n * C + c] * inv;
        dx[i] = acc ? dx[i] + v : v;
    }
}

// ---- per-channel column reductions ----------------------------------------
// Workgroup (bx, by): channels [bx*64, bx*64+64), rows [by*RB, by*RB+RB).
// 256 threads = 64 channels x 4 row lanes; the 4 row-lane sums are combined
// in LDS in a fixed order.
constexpr int CS_CH = 64;
constexpr int CS_RB = 256;

inline int cs_row_blocks(long M) { return (int)((M + CS_RB - 1) / CS_RB); }

// mode 0: sum v;  mode 1: sum (v - mean[c])^2;  mode 2: sum dy', sum dy'*xhat
// (two outputs) where dy' = dy masked by relu_y > 0 if relu_y is given.
template <int MODE>
__global__ void colsum_partial_kernel(const float* __restrict__ v, const float* __restrict__ x,
                                      const float* __restrict__ relu_y,
                                      const float* __restrict__ mean,
                                      const float* __restrict__ invstd, long M, int C,
                                      float* __restrict__ part0, float* __restrict__ part1) {
    __shared__ float red0[4][CS_CH];
    __shared__ float red1[4][CS_CH];
    const int cl = threadIdx.x % CS_CH;
    const int rl = threadIdx.x / CS_CH;
    const int c = blockIdx.x * CS_CH + cl;
    const long r0 = (long)blockIdx.y * CS_RB;
    const long r1 = min(r0 + CS_RB, M);
    float s0 = 0.f, s1 = 0.f;
    if (c < C) {
        float mu = 0.f, is = 0.f;
        if (MODE >= 1) mu = mean[c];
        if (MODE == 2) is = invstd[c];
        for (long r = r0 + rl; r < r1; r += 4) {
            size_t idx = (size_t)r * C + c;
            if (MODE == 0) {
                s0 += v[idx];
            } else if (MODE == 1) {
                float d = v[idx] - mu;
                s0 += d * d;
            } else {
                float g = v[idx];
                if (relu_y && !(relu_y[idx] > 0.f)) g = 0.f;
                float xh = (x[idx] - mu) * is;
                s0 += g;
                s1 += g * xh;
            }
        }
    }
    red0[rl][cl] = s0;
    red1[rl][cl] = s1;
    __syncthreads();
    if (rl == 0 && c < C) {
        float a0 = ((red0[0][cl] + red0[1][cl]) + red0[2][cl]) + red0[3][cl];
        part0[(size_t)blockIdx.y * C + c] = a0;
        if (MODE == 2) {
            float a1 = ((red1[0][cl] + red1[1][cl]) + red1[2][cl]) + red1[3][cl];
            part1[(size_t)blockIdx.y * C + c] = a1;
        }
    }
}

// Final reduction of the row-block partials: workgroup = 64 channels x 16
// lanes; lane l sums partial rows l, l+16, ...; the 16 lane sums are combined
// in LDS in a fixed order.  mode 0: out = sum; 1: out = sum / M (mean);
// 2: out = 1 / sqrt(sum / M + eps) (inverse standard deviation).
constexpr int CF_LANES = 16;

__global__ void colsum_final_kernel(const float* __restrict__ part, int nb, int C, long M,
                                    float eps, int mode, float* __restrict__ out) {
    __shared__ float red[CF_LANES][CS_CH];
    const int cl = threadIdx.x % CS_CH;
    const int rl = threadIdx.x / CS_CH;
    const int c = blockIdx.x * CS_CH + cl;
    float s = 0.f;
    if (c < C)
        for (int b = rl; b < nb; b += CF_LANES) s += part[(size_t)b * C + c];
    red[rl][cl] = s;
    __syncthreads();
    if (rl == 0 && c < C) {
        float t = 0.f;
        for (int l = 0; l < CF_LANES; ++l) t += red[l][cl];
        if (mode == 1) t = t / (float)M;
        else if (mode == 2) t = 1.f / sqrtf(t / (float)M + eps);
        out[c] = t;
    }
}

__global__ void bn_apply_kernel(const float* __restrict__ x, long M, int C,
                                const float* __restrict__ gamma, const float* __restrict__ beta,
                                const float* __restrict__ mean, const float* __restrict__ invstd,
                                float* __restrict__ y, int relu) {
    const size_t total = (size_t)M * C;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        float v = gamma[c] * ((x[i] - mean[c]) * invstd[c]) + beta[c];
        y[i] = relu ? fmaxf(v, 0.f) : v;
    }
}

// dx = gamma*invstd*(dy' - sdy/M - xhat*sdyx/M)
__global__ void bn_bwd_apply_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                    const float* __restrict__ relu_y, long M, int C,
                                    const float* __restrict__ gamma,
                                    const float* __restrict__ mean,
                                    const float* __restrict__ invstd,
                                    const float* __restrict__ sdy, const float* __restrict__ sdyx,
                                    float* __restrict__ dx, int acc) {
    const size_t total = (size_t)M * C;
    const float invM = 1.f / (float)M;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        int c = (int)(i % C);
        float g = dy[i];
        if (relu_y && !(relu_y[i] > 0.f)) g = 0.f;
        float is = invstd[c];
        float xh = (x[i] - mean[c]) * is;
        float v = gamma[c] * is * (g - sdy[c] * invM - xh * (sdyx[c] * invM));
        dx[i] = acc ? dx[i] + v : v;
    }
}

// softmax cross-entropy: one workgroup per row
__global__ void softmax_ce_kernel(const float* __restrict__ z, const int32_t* __restrict__ labels,
                                  int B, int K, float* __restrict__ row_loss,
                                  float* __restrict__ dz) {
    __shared__ float red[EW_THREADS];
    const int n = blockIdx.x;
    const float* zr = z + (size_t)n * K;
    float m = -INFINITY;
    for (int k = threadIdx.x; k < K; k += blockDim.x) m = fmaxf(m, zr[k]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int o = EW_THREADS / 2; o > 0; o >>= 1) {
        if (threadIdx.x < o) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + o]);
        __syncthreads();
    }
    m = red[0];
    __syncthreads();
    float s = 0.f;
    for (int k = threadIdx.x; k < K; k += blockDim.x) s += expf(zr[k] - m);
    red[threadIdx.x] = s;
    __syncthreads();
    for (int o = EW_THREADS / 2; o > 0; o >>= 1) {
        if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
        __syncthreads();
    }
    const float lse = m + logf(red[0]);
    const int lab = labels[n];
    const bool lab_ok = lab >= 0 && lab < K;   // an invalid label yields a NaN loss, no fault
    const float invB = 1.f / (float)B;
    for (int k = threadIdx.x; k < K; k += blockDim.x) {
        float p = expf(zr[k] - lse);
        dz[(size_t)n * K + k] = (p - (k == lab ? 1.f : 0.f)) * invB;
    }
    if (threadIdx.x == 0) row_loss[n] = lab_ok ? lse - zr[lab] : __builtin_nanf("");
}

__global__ void mean_rows_kernel(const float* __restrict__ row_loss, int B,
                                 float* __restrict__ loss) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        float s = 0.f;
        for (int n = 0; n < B; ++n) s += row_loss[n];
        *loss = s / (float)B;
    }
}

}  // namespace

hipError_t launch_relu_fwd(const float* x, float* y, size_t n, hipStream_t s) {
    hipLaunchKernelGGL(relu_fwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, y, n);
    return hipGetLastError();
}

hipError_t launch_relu_bwd(const float* y, const float* dy, float* dx, size_t n, int accumulate,
                           hipStream_t s) {
    hipLaunchKernelGGL(relu_bwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, y, dy, dx, n,
                       accumulate);
    return hipGetLastError();
}

hipError_t launch_add_fwd(const float* a, const float* b, float* y, size_t n, int relu,
                          hipStream_t s) {
    hipLaunchKernelGGL(add_fwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, a, b, y, n,
                       relu);
    return hipGetLastError();
}

hipError_t launch_copy_or_acc(const float* v, float* out, size_t n, int accumulate,
                              hipStream_t s) {
    hipLaunchKernelGGL(copy_or_acc_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, v, out, n,
                       accumulate);
    return hipGetLastError();
}

hipError_t launch_maxpool_fwd(const float* x, float* y, int N, int H, int W, int C, int R, int S,
                              int st, int pad, int P, int Q, hipStream_t s) {
    size_t n = (size_t)N * P * Q * C;
    hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, y, N, H,
                       W, C, R, S, st, pad, P, Q);
    return hipGetLastError();
}

hipError_t launch_maxpool_bwd(const float* x, const float* dy, float* dx, int N, int H, int W,
                              int C, int R, int S, int st, int pad, int P, int Q, int accumulate,
                              const float* mask, hipStream_t s) {
    if (R == S && R == st && pad == 0 && P * st == H && Q * st == W) {
        size_t n = (size_t)N * P * Q * C;
        if (R == 2)
            hipLaunchKernelGGL(maxpool_bwd_tiled_kernel<2>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0,
                               s, x, dy, dx, N, H, W, C, R, P, Q, accumulate, mask);
        else
            hipLaunchKernelGGL(maxpool_bwd_tiled_kernel<0>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0,
                               s, x, dy, dx, N, H, W, C, R, P, Q, accumulate, mask);
        return hipGetLastError();
    }
    size_t n = (size_t)N * H * W * C;
    hipLaunchKernelGGL(maxpool_bwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, dy, dx,
                       N, H, W, C, R, S, st, pad, P, Q, accumulate, mask);
    return hipGetLastError();
}

hipError_t launch_gap_fwd(const float* x, float* y, int N, int HW, int C, hipStream_t s) {
    size_t n = (size_t)N * C;
    hipLaunchKernelGGL(gap_fwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, y, N, HW, C);
    return hipGetLastError();
}

hipError_t launch_gap_bwd(const float* dy, float* dx, int N, int HW, int C, int accumulate,
                          hipStream_t s) {
    size_t n = (size_t)N * HW * C;
    hipLaunchKernelGGL(gap_bwd_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, dy, dx, N, HW,
                       C, accumulate);
    return hipGetLastError();
}

size_t colsum_ws_floats(long M, int C) { return (size_t)cs_row_blocks(M) * C; }

hipError_t launch_colsum(const float* v, long M, int C, float* out, float* ws, hipStream_t s) {
    int nb = cs_row_blocks(M);
    dim3 grid((C + CS_CH - 1) / CS_CH, nb);
    hipLaunchKernelGGL(colsum_partial_kernel<0>, grid, dim3(256), 0, s, v, nullptr, nullptr,
                       nullptr, nullptr, M, C, ws, nullptr);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + CS_CH - 1) / CS_CH), dim3(CS_CH * CF_LANES), 0,
                       s, ws, nb, C, M, 0.f, 0, out);
    return hipGetLastError();
}

size_t bn_ws_floats(long M, int C) { return 2 * (size_t)cs_row_blocks(M) * C + 2 * (size_t)C; }

hipError_t launch_bn_fwd(const float* x, long M, int C, const float* gamma, const float* beta,
                         float eps, float* y, float* mean, float* invstd, int relu, float* ws,
                         hipStream_t s) {
    int nb = cs_row_blocks(M);
    dim3 grid((C + CS_CH - 1) / CS_CH, nb);
    hipLaunchKernelGGL(colsum_partial_kernel<0>, grid, dim3(256), 0, s, x, nullptr, nullptr,
                       nullptr, nullptr, M, C, ws, nullptr);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + CS_CH - 1) / CS_CH), dim3(CS_CH * CF_LANES), 0,
                       s, ws, nb, C, M, 0.f, 1, mean);
    hipLaunchKernelGGL(colsum_partial_kernel<1>, grid, dim3(256), 0, s, x, nullptr, nullptr, mean,
                       nullptr, M, C, ws, nullptr);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + CS_CH - 1) / CS_CH), dim3(CS_CH * CF_LANES), 0,
                       s, ws, nb, C, M, eps, 2, invstd);
    size_t n = (size_t)M * C;
    hipLaunchKernelGGL(bn_apply_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, M, C, gamma,
                       beta, mean, invstd, y, relu);
    return hipGetLastError();
}

hipError_t launch_bn_bwd(const float* x, const float* dy, const float* relu_y, long M, int C,
                         const float* gamma, const float* mean, const float* invstd, float* dx,
                         float* dgamma, float* dbeta, int accumulate, float* ws, hipStream_t s) {
    int nb = cs_row_blocks(M);
    float* p0 = ws;
    float* p1 = ws + (size_t)nb * C;
    dim3 grid((C + CS_CH - 1) / CS_CH, nb);
    hipLaunchKernelGGL(colsum_partial_kernel<2>, grid, dim3(256), 0, s, dy, x, relu_y, mean,
                       invstd, M, C, p0, p1);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + CS_CH - 1) / CS_CH), dim3(CS_CH * CF_LANES), 0,
                       s, p0, nb, C, M, 0.f, 0, dbeta);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + CS_CH - 1) / CS_CH), dim3(CS_CH * CF_LANES), 0,
                       s, p1, nb, C, M, 0.f, 0, dgamma);
    if (!dx) return hipGetLastError();      // parameter gradients only
    size_t n = (size_t)M * C;
    hipLaunchKernelGGL(bn_bwd_apply_kernel, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, dy,
                       relu_y, M, C, gamma, mean, invstd, dbeta, dgamma, dx, accumulate);
    return hipGetLastError();
}

hipError_t launch_softmax_ce(const float* z, const int32_t* labels, int B, int K, float* loss,
                             float* dz, float* ws, hipStream_t s) {
    hipLaunchKernelGGL(softmax_ce_kernel, dim3(B), dim3(EW_THREADS), 0, s, z, labels, B, K, ws, dz);
    hipLaunchKernelGGL(mean_rows_kernel, dim3(1), dim3(64), 0, s, ws, B, loss);
    return hipGetLastError();
}

}  // namespace hp
