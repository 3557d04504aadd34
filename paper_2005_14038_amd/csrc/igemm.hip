// Implicit-GEMM convolution / FC contractions on CDNA4 MFMA (gfx950).
//
// One kernel template per precision covers the three contractions of a
// convolution layer (an FC layer is a 1x1 convolution on a 1x1 map):
//
//   forward  out[m = (n,p,q)][k]     = sum_{(r,s,c)} x[n, p*st-pad+r, q*st-pad+s, c] w[k,r,s,c]
//   dgrad    out[m = (n,h,w)][c]     = sum_{(r,s,k)} dy[n, (h+pad-r)/st, (w+pad-s)/st, k] w[k,r,s,c]
//                                      (only taps where the division is exact and in range)
//   wgrad    out[k][j = (r,s,c)]     = sum_{(n,p,q)} dy[n,p,q,k] x[n, p*st-pad+r, q*st-pad+s, c]
//
// The operands are gathered straight from the NHWC activations and the KRSC
// weights ("implicit" im2col: nothing is materialised), staged through LDS,
// double buffered, and fed to the matrix cores; each wave64 owns a WM x WN
// block of the output as a grid of MFMA 32x32 tiles.
//
//   fp32: v_mfma_f32_32x32x2_f32; LDS tiles [BK][rows] (row index contiguous).
//   bf16: every operand is rounded to bfloat16 (RNE), either as it is staged
//         from fp32 or once, into a bf16 copy in memory, by the layer that
//         produces it; v_mfma_f32_32x32x16_bf16 reads LDS tiles of BKH = 32
//         or 64 reduction indices per row.  Products of bf16 values are exact
//         in fp32 and the accumulation stays fp32.  Kernels: general gather
//         (igemm_bf16_kernel from fp32, igemm_h16_kernel from bf16), buffer
//         loads for k-major operands (igemm_h16k_kernel: forward, data
//         gradient) and m-major LDS tiles with transpose reads
//         (igemm_h16w_kernel: weight gradient).
//
// Long reductions (weight gradients reduce over N*P*Q, FC layers over their
// fan-in) and layers with too few output tiles to fill the chip are cut into
// chunks; each chunk writes a partial tile to a workspace and a second kernel
// adds the partials in a fixed order, so results are deterministic.
#include <type_traits>

#include "kernels.h"

namespace hp {

typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

// LDS row padding (floats).  Operands staged from k-major rows are written
// transposed, one float per store: a row length of 2 mod 32 spreads a wave's
// stores over distinct banks.  Operands staged as whole float4 rows need a
// row length that keeps 16-byte alignment.
constexpr int PAD_T = 2;
constexpr int PAD_V = 4;

// Tile configurations: workgroup tile BM x BN, reduction tile BK of the
// kernels that stage from fp32 and BKH of the kernels on bf16 operands in
// memory, wave tile WM x WN (a grid of (WM/32) x (WN/32) MFMA 32x32 tiles per
// wave); the workgroup has (BM/WM) * (BN/WN) waves.  BKH = 64 halves the
// barriers per MFMA; the 128x64 tile keeps 32, where the second register set
// of a 64-wide k tile would cost it occupancy.
struct TileCfg { int bm, bn, bk, wm, wn, bkh; };
// Waves of 32x64 (eight in the general tile, four in the 128x64 and 64x128
// ones) hide the staging latency better than fewer waves of 64x64, at the
// cost of more LDS reads per MFMA.
constexpr TileCfg kCfgs[] = {
    {128, 128, 16, 32, 64, 64},    // 0: general (8 waves)
    {128, 64, 16, 32, 64, 32},     // 1: narrow N (at most 64 output columns, 4 waves)
    {64, 256, 16, 64, 64, 32},     // 2: narrow M, N a multiple of 256 or large
    {64, 128, 16, 32, 64, 64},     // 3: narrow M otherwise (4 waves)
    {64, 64, 16, 32, 32, 64},      // 4: small M and N (4 waves of 32x32)
    {256, 128, 16, 128, 64, 32},   // 5: igemm_h16d_kernel (4 waves)
};

struct KArgs {
    ConvGeo g;
    const float* a;
    const float* b;
    float* out;
    const float* bias;
    const float* mask;
    float* bias_out;
    long M, Ncols, Kred;
    int tiles_m, tiles_n;
    int tfull;        // tiles computed whole, one per workgroup (the first tfull ids)
    int splits;       // every remaining tile is cut into `splits` reduction chunks
    int kchunk;       // reduction length of a chunk (multiple of the K tile)
    float* ws;        // partial tiles of the cut tiles: [tile - tfull][split][BM * BN]
    float* stats;     // optional column statistics per row tile (see Epilogue)
    int epi;
    const unsigned short* a16;   // bf16 copies of a and b (16-bit operand kernel only)
    const unsigned short* b16;
    // optional: every final output element is also written here rounded to
    // bf16 (nearest even), row-major like out (no bias-gradient column)
    unsigned short* out16;
    // weight gradient on bf16 operands: floor(i / Q) = (i * mq) >> sq and
    // floor(i / P) = (i * mp) >> sp for 0 <= i < 2^31
    unsigned mq, mp;
    int sq, sp;
};

// Destination of output element (row, col): the bias-gradient column of a
// weight gradient goes to bias_out[row]; everything else is row-major with
// the weight part's row length.
__device__ __forceinline__ float* out_ptr(float* out, float* bias_out, long row, long col,
                                          long Ncols, int epi) {
    if (epi & EPI_BIASCOL) {
        if (col == Ncols - 1) return bias_out + row;
        return out + row * (Ncols - 1) + col;
    }
    return out + row * Ncols + col;
}

__device__ __forceinline__ float epilogue(float v, long row, long col, long Ncols, int epi,
                                          const float* bias, const float* mask, const float* prev) {
    if (epi & EPI_BIAS) v += bias[col];
    if (epi & EPI_RELU) v = fmaxf(v, 0.f);
    if ((epi & EPI_MASK) && !(mask[row * Ncols + col] > 0.f)) v = 0.f;
    if (epi & EPI_ACCUM) v += *prev;
    return v;
}

__device__ __forceinline__ float round_bf16(float x) {
    unsigned u = __float_as_uint(x);
    u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
    return __uint_as_float(u);
}

// Two floats rounded to bf16, packed low element first (LDS byte order).
__device__ __forceinline__ unsigned pack_bf16(float lo, float hi) {
    return (__float_as_uint(round_bf16(lo)) >> 16) | (__float_as_uint(round_bf16(hi)) & 0xFFFF0000u);
}

__device__ __forceinline__ unsigned short bf16_bits(float x) {
    return (unsigned short)(__float_as_uint(round_bf16(x)) >> 16);
}

// Work assignment.  The first `tfull` workgroups each compute one whole
// output tile (whole rounds of the resident workgroups); the rest cut each
// remaining tile's reduction into `splits` chunks, so that the last round is
// as full as the others, and leave partial tiles for the reduce kernels.
// XCD-aware: consecutive workgroup ids are dealt round-robin to the 8 XCDs;
// each XCD gets a contiguous run of whole tiles (n fastest), so tiles sharing
// A rows share that XCD's L2, and likewise a contiguous run of cut-tile items
// (chunk, tile), so tiles reducing over the same chunk share it.
struct Work {
    int tile, z;
    bool partial;
    long m0, n0, kbeg, kend;
};

template <int BM, int BN>
__device__ __forceinline__ Work decode_work(const KArgs& args) {
    Work w;
    int bid = blockIdx.x;
    w.z = 0;
    w.partial = bid >= args.tfull;
    if (!w.partial) {
        if ((args.tfull & 7) == 0) bid = (bid & 7) * (args.tfull >> 3) + (bid >> 3);
        w.tile = bid;
    } else {
        const int r = bid - args.tfull;
        const int ncut = args.tiles_m * args.tiles_n - args.tfull;
        if ((args.tfull & 7) == 0) {
            // the workgroups of one XCD (ids congruent mod 8) take a contiguous
            // run of (chunk, tile) items, tiles fastest: the cut tiles that
            // reduce over the same chunk (same dy rows, same image rows) share
            // that XCD's L2
            const int nparts = ncut * args.splits;
            const int x = r & 7, q = nparts >> 3, rem = nparts & 7;
            const int item = x * q + min(x, rem) + (r >> 3);
            w.z = item / ncut;
            w.tile = args.tfull + (item - w.z * ncut);
        } else {
            w.tile = args.tfull + r / args.splits;
            w.z = r - (w.tile - args.tfull) * args.splits;
        }
    }
    w.m0 = (long)(w.tile / args.tiles_n) * BM;
    w.n0 = (long)(w.tile % args.tiles_n) * BN;
    w.kbeg = w.partial ? (long)w.z * args.kchunk : 0;
    w.kend = w.partial ? min(w.kbeg + (long)args.kchunk, args.Kred) : args.Kred;
    return w;
}

// Writes a wave's accumulators: acc[i][j][v] holds
// out[m0 + wm + 32i + 8(v/4) + 4(lane/32) + v%4][n0 + wn + 32j + lane%32]
// (the output layout of the 32x32 MFMAs), through the epilogue, or raw into
// the workspace slot of a cut tile.  The epilogue's reads (the previous
// output to accumulate into, the ReLU mask) of one 32x32 tile are all issued
// before its stores: a store may alias a later read as far as the compiler
// knows, so interleaving them would serialise one memory latency per element.
constexpr int EPI_CHUNK = 8;     // outputs per lane whose epilogue reads are batched

template <int BM, int BN, int TM, int TN, bool FENCE = false>
__device__ __forceinline__ void store_tile(const KArgs& args, const Work& w,
                                           const floatx16 (&acc)[TM][TN], int wm, int wn,
                                           int lane) {
    const int lr = lane & 31, lk = lane >> 5;
    if (w.partial) {
        float* pslot = args.ws + ((long)(w.tile - args.tfull) * args.splits + w.z) * (BM * BN);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
                if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);   // one block at a time
            const int lcol = wn + 32 * j + lr;
            if (w.n0 + lcol >= args.Ncols) continue;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int lrow = wm + 32 * i + 8 * (v >> 2) + 4 * lk + (v & 3);
                    if (w.m0 + lrow < args.M) pslot[lrow * BN + lcol] = acc[i][j][v];
                }
        }
        return;
    }
    const int epi = args.epi;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const long col = w.n0 + wn + 32 * j + lr;
        if (col >= args.Ncols) continue;
        // output row stride and the address of (row0, col); the bias-gradient
        // column goes to bias_out[row]
        long ld = args.Ncols;
        float* cbase = args.out + col;
        if (epi & EPI_BIASCOL) {
            ld = args.Ncols - 1;
            cbase = args.out + col;
            if (col == args.Ncols - 1) { ld = 1; cbase = args.bias_out; }
        }
        const float bias = (epi & EPI_BIAS) ? args.bias[col] : 0.f;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);   // one block at a time
            const long row0 = w.m0 + wm + 32 * i + 4 * lk;
            // rows row0 + 8(v/4) + v%4 of this lane; those >= M are outside
            const int left = (int)min(args.M - row0, 32L);
            float* obase = cbase + row0 * ld;
            const float* mbase = (epi & EPI_MASK) ? args.mask + row0 * args.Ncols + col : nullptr;
            const int ldi = (int)ld, ldm = (int)args.Ncols;
#pragma unroll
            for (int v0 = 0; v0 < 16; v0 += EPI_CHUNK) {
                float prev[EPI_CHUNK], msk[EPI_CHUNK];
#pragma unroll
                for (int u = 0; u < EPI_CHUNK; ++u) {
                    const int r = 8 * ((v0 + u) >> 2) + ((v0 + u) & 3);
                    prev[u] = 0.f;
                    msk[u] = 1.f;
                    if (r < left) {
                        if (epi & EPI_ACCUM) prev[u] = obase[r * ldi];
                        if (epi & EPI_MASK) msk[u] = mbase[r * ldm];
                    }
                }
#pragma unroll
                for (int u = 0; u < EPI_CHUNK; ++u) {
                    const int r = 8 * ((v0 + u) >> 2) + ((v0 + u) & 3);
                    if (r >= left) continue;
                    float val = acc[i][j][v0 + u];
                    if (epi & EPI_BIAS) val += bias;
                    if (epi & EPI_RELU) val = fmaxf(val, 0.f);
                    if ((epi & EPI_MASK) && !(msk[u] > 0.f)) val = 0.f;
                    if (epi & EPI_ACCUM) val += prev[u];
                    obase[r * ldi] = val;
                    if (args.out16) args.out16[(row0 + r) * args.Ncols + col] = bf16_bits(val);
                }
            }
        }
    }
}

// The same writes through the wave's private 4 KB LDS slot (the k loop's
// buffers are free once its last barrier has passed): each 32x32 block is
// staged in LDS and read back with every lane holding 4 consecutive columns of
// one row (8 rows per pass, 4 passes, two at a time), so the epilogue's loads and stores are
// 16 bytes wide instead of 4.  Used when the output, the bias and the mask
// allow 16-byte access and there is no bias-gradient column; a group of 4
// columns that crosses the last column is written element by element.
constexpr int SLOT_FLOATS = 32 * 32;

template <int BM, int BN, int TM, int TN, bool FENCE = false>
__device__ __forceinline__ void store_tile_wide(const KArgs& args, const Work& w,
                                                const floatx16 (&acc)[TM][TN], int wm, int wn,
                                                int lane, float* slot) {
    const int lr = lane & 31, lk = lane >> 5;
    const int rq = lane >> 3, cq = (lane & 7) * 4;
    const int epi = args.epi;
    const long N = args.Ncols;
    float* pslot =
        w.partial ? args.ws + ((long)(w.tile - args.tfull) * args.splits + w.z) * (BM * BN)
                  : nullptr;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);   // one block at a time
#pragma unroll
            for (int v = 0; v < 16; ++v)
                slot[(8 * (v >> 2) + 4 * lk + (v & 3)) * 32 + lr] = acc[i][j][v];
            const int lcol = wn + 32 * j + cq;
            const long col = w.n0 + lcol;
            const bool full = col + 3 < N;
            float4 bias = make_float4(0.f, 0.f, 0.f, 0.f);
            if (!w.partial && (epi & EPI_BIAS) && col < N) {
                if (full) {
                    bias = *reinterpret_cast<const float4*>(args.bias + col);
                } else {
                    bias.x = args.bias[col];
                    if (col + 1 < N) bias.y = args.bias[col + 1];
                    if (col + 2 < N) bias.z = args.bias[col + 2];
                }
            }
            // two passes (rows 8q + rq) at a time: their epilogue reads first,
            // then the stores
#pragma unroll
            for (int q0 = 0; q0 < 4; q0 += 2) {
                float4 val[2];
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    val[h] = *reinterpret_cast<const float4*>(slot + (8 * (q0 + h) + rq) * 32 + cq);
                if (w.partial) {
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int lrow = wm + 32 * i + 8 * (q0 + h) + rq;
                        if (w.m0 + lrow < args.M && col < N)
                            *reinterpret_cast<float4*>(pslot + lrow * BN + lcol) = val[h];
                    }
                    continue;
                }
                if (col >= N) continue;
                float4 prev[2], msk[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const long row = w.m0 + wm + 32 * i + 8 * (q0 + h) + rq;
                    prev[h] = make_float4(0.f, 0.f, 0.f, 0.f);
                    msk[h] = make_float4(1.f, 1.f, 1.f, 1.f);
                    if (row >= args.M) continue;
                    const long off = row * N + col;
                    if (full) {
                        if (epi & EPI_ACCUM) prev[h] = *reinterpret_cast<const float4*>(args.out + off);
                        if (epi & EPI_MASK) msk[h] = *reinterpret_cast<const float4*>(args.mask + off);
                    } else {
                        float* pp = &prev[h].x;
                        float* mm = &msk[h].x;
                        for (int e = 0; e < 4 && col + e < N; ++e) {
                            if (epi & EPI_ACCUM) pp[e] = args.out[off + e];
                            if (epi & EPI_MASK) mm[e] = args.mask[off + e];
                        }
                    }
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const long row = w.m0 + wm + 32 * i + 8 * (q0 + h) + rq;
                    if (row >= args.M) continue;
                    float o[4] = {val[h].x, val[h].y, val[h].z, val[h].w};
                    const float b4[4] = {bias.x, bias.y, bias.z, bias.w};
                    const float p4[4] = {prev[h].x, prev[h].y, prev[h].z, prev[h].w};
                    const float m4[4] = {msk[h].x, msk[h].y, msk[h].z, msk[h].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if (epi & EPI_BIAS) o[e] += b4[e];
                        if (epi & EPI_RELU) o[e] = fmaxf(o[e], 0.f);
                        if ((epi & EPI_MASK) && !(m4[e] > 0.f)) o[e] = 0.f;
                        if (epi & EPI_ACCUM) o[e] += p4[e];
                    }
                    const long off = row * N + col;
                    if (full) {
                        *reinterpret_cast<float4*>(args.out + off) =
                            make_float4(o[0], o[1], o[2], o[3]);
                        if (args.out16) {
                            uint2 h;
                            h.x = pack_bf16(o[0], o[1]);
                            h.y = pack_bf16(o[2], o[3]);
                            *reinterpret_cast<uint2*>(args.out16 + off) = h;
                        }
                    } else {
                        for (int e = 0; e < 4 && col + e < N; ++e) {
                            args.out[off + e] = o[e];
                            if (args.out16) args.out16[off + e] = bf16_bits(o[e]);
                        }
                    }
                }
            }
        }
    }
}

// Column statistics of a whole tile for a following batch norm: the mean of
// each column over the tile's rows below M and the sum of squared deviations
// from it, two passes over the accumulators (values after the bias), lanes l
// and l + 32 combined by a shuffle, the waves along M through LDS in a fixed
// order.  Every thread of the workgroup takes part (barriers); lds holds at
// least (BM / WM + 1) * BN floats.
template <int BM, int BN, int TM, int TN>
__device__ __forceinline__ void tile_stats(const KArgs& args, const Work& w,
                                           const floatx16 (&acc)[TM][TN], int wm, int wn,
                                           int lane, float* lds) {
    constexpr int WAVES_M = BM / (32 * TM);
    const int lr = lane & 31, lk = lane >> 5;
    const int wave_m = wm / (32 * TM);
    const long rows = min((long)BM, args.M - w.m0);
    float* part = lds;                   // [WAVES_M][BN]
    float* mean = lds + WAVES_M * BN;    // [BN]
    const int t = threadIdx.x;
    const int nthreads = blockDim.x;
    float bias[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const long col = w.n0 + wn + 32 * j + lr;
        bias[j] = ((args.epi & EPI_BIAS) && col < args.Ncols) ? args.bias[col] : 0.f;
    }
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const float mu = pass ? mean[wn + 32 * j + lr] : 0.f;
            float sum = 0.f;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int r = wm + 32 * i + 8 * (v >> 2) + 4 * lk + (v & 3);
                    if (r < rows) {
                        const float d = acc[i][j][v] + bias[j] - mu;
                        sum += pass ? d * d : d;
                    }
                }
            sum += __shfl_xor(sum, 32);
            if (lk == 0) part[wave_m * BN + wn + 32 * j + lr] = sum;
        }
        __syncthreads();
        for (int c = t; c < BN; c += nthreads) {
            float s = 0.f;
            for (int m = 0; m < WAVES_M; ++m) s += part[m * BN + c];
            const long col = w.n0 + c;
            if (pass == 0) {
                mean[c] = rows > 0 ? s / (float)rows : 0.f;
            } else if (col < args.Ncols) {
                const long tm = w.m0 / BM;
                args.stats[tm * args.Ncols + col] = mean[c];
                args.stats[((long)args.tiles_m + tm) * args.Ncols + col] = s;
            }
        }
        __syncthreads();
    }
}

// Writes a wave's tile: the wide path when the kernel was built with it
// (WIDE) and its conditions hold (uniform).  The wide path costs registers,
// which the fp32 kernels on long reductions, where the epilogue is a small
// part of the time, keep for occupancy.
// The epilogue without column statistics: the wide path where the output, the
// bias, the mask and the workspace allow 16-byte access and there is no
// bias-gradient column, else the narrow one.
template <int BM, int BN, int TM, int TN, bool FENCE = false>
__device__ __forceinline__ void write_tile_plain(const KArgs& args, const Work& w,
                                                 const floatx16 (&acc)[TM][TN], int wm, int wn,
                                                 int lane, float* slot) {
    auto a16 = [](const void* p) { return (((uintptr_t)p) & 15) == 0; };
    const int epi = args.epi;
    const bool wide = !(epi & EPI_BIASCOL) && (args.Ncols & 3) == 0 && a16(args.out) &&
                      (!(epi & EPI_BIAS) || a16(args.bias)) &&
                      (!(epi & EPI_MASK) || a16(args.mask)) && a16(args.ws);
    if (wide)
        store_tile_wide<BM, BN, TM, TN, FENCE>(args, w, acc, wm, wn, lane, slot);
    else
        store_tile<BM, BN, TM, TN, FENCE>(args, w, acc, wm, wn, lane);
}

template <int BM, int BN, int TM, int TN, bool WIDE = true>
__device__ __forceinline__ void write_tile(const KArgs& args, const Work& w,
                                           const floatx16 (&acc)[TM][TN], int wm, int wn,
                                           int lane, float* slot, float* lds_all) {
    if constexpr (WIDE) {
        // column statistics of whole tiles (uniform per workgroup: it is either
        // whole or cut); the LDS slots are reused afterwards.  Built only into
        // the wide kernels, whose register budget already allows it.
        if (args.stats && !w.partial)
            tile_stats<BM, BN, TM, TN>(args, w, acc, wm, wn, lane, lds_all);
        write_tile_plain<BM, BN, TM, TN>(args, w, acc, wm, wn, lane, slot);
        return;
    }
    store_tile<BM, BN, TM, TN>(args, w, acc, wm, wn, lane);
}

// Raw buffer loads: the hardware's range check returns zeros for an offset at
// or past the end of the buffer, so an operand element that lies in the
// padding or outside the matrix is read with an offset of BUF_OOB instead of
// being masked.
typedef unsigned uintx4 __attribute__((ext_vector_type(4)));
constexpr unsigned BUF_OOB = 0x80000000u;      // buffer offset past any operand here
constexpr int BUF_CFG = 0x00020000;            // buffer descriptor word 3 (gfx9 family)

__device__ __forceinline__ uintx4 buf_load16(__amdgpu_buffer_rsrc_t rs, unsigned voff,
                                             unsigned soff) {
    return __builtin_amdgcn_raw_buffer_load_b128(rs, (int)voff, (int)soff, 0);
}

// ---- operand gathers -------------------------------------------------------
// Each returns VW consecutive elements along the operand's contiguous axis
// (zero where the element lies outside the problem or in the padding).

template <int VW>
__device__ __forceinline__ void load_vec(const float* p, bool ok, float* v) {
    if constexpr (VW == 4) {
        if (ok) {
            float4 t = *reinterpret_cast<const float4*>(p);
            v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
        } else {
            v[0] = v[1] = v[2] = v[3] = 0.f;
        }
    } else {
        v[0] = ok ? *p : 0.f;
    }
}

// FAST: a forward or stride-1 data-gradient contraction whose reduction
// channel count (C, or K) is a multiple of the k tile, with the tap-inner
// order and the unit stride fixed at compile time: no k tile crosses a tap,
// so the per-thread wrap of the channel index, the linear-order paths and the
// stride's division and exact-tap test drop out of the k loop (the data
// gradient's stride alone: VGG-19 +1.1 %, its first stage +1.3 %).  The tap
// index steps by selects and (r, s) follow from it by a multiply and shift,
// exact for at most 7 x 7 taps (the host's condition).  For a
// weight gradient: an output width Q that is a multiple of the k tile, so that
// no k tile (16 output pixels) crosses an output row and the pixel's image
// and row are the tile's.
template <int OP, int BM, int BN, int BK, int WM, int WN, int VW, bool WIDE = false,
          bool FAST = false>
__global__ void __launch_bounds__(64 * (BM / WM) * (BN / WN), 2) igemm_kernel(KArgs args) {
    constexpr int NT = 64 * (BM / WM) * (BN / WN);
    constexpr int TM = WM / 32, TN = WN / 32;  // MFMA tiles per wave
    constexpr bool A_KMAJ = (OP != OP_WGRAD);
    constexpr bool B_KMAJ = (OP == OP_FWD);
    constexpr int LDA = BM + (A_KMAJ ? PAD_T : PAD_V);
    constexpr int LDB = BN + (B_KMAJ ? PAD_T : PAD_V);
    constexpr int WAVES_N = BN / WN;
    __shared__ float smem[2 * BK * (LDA + LDB)];

    const ConvGeo& g = args.g;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int wm = (wave / WAVES_N) * WM;
    const int wn = (wave % WAVES_N) * WN;

    const Work wk = decode_work<BM, BN>(args);
    const long m0 = wk.m0, n0 = wk.n0, kbeg = wk.kbeg, kend = wk.kend;
    const int ktiles = (int)((kend - kbeg + BK - 1) / BK);

    // Reduction order of the k tiles.  When the channel count of a tap is a
    // multiple of BK (every tile lies within one tap) the tiles are taken
    // channel chunk by channel chunk, all taps of a chunk in a row: the R*S
    // tap-shifted reads of the same BK channels follow each other and hit in
    // the caches instead of coming back from DRAM once per tap.  Tile T is
    // then (chunk T / RS, tap T % RS); a cut chunk covers a range of T.
    // Otherwise tiles follow the linear reduction index.
    const int CCH = (OP == OP_FWD) ? g.C : g.K;
    const int RSN = g.R * g.S;
    const bool tap_inner = (OP != OP_WGRAD) && (FAST || ((CCH % BK == 0) && RSN > 1));
    const int tbeg = (int)(kbeg / BK), tend = (int)((kend + BK - 1) / BK);

    // ---- per-thread staging coordinates ----
    // A: OP_FWD / OP_DGRAD gather rows m with the reduction index contiguous
    // ("k-major"); OP_WGRAD reads dy rows (reduction index = row) with m = k
    // contiguous ("m-major").  B: OP_FWD reads weight rows (k-major);
    // OP_DGRAD / OP_WGRAD read rows indexed by the reduction with n contiguous.
    constexpr int AV = A_KMAJ ? (BM * BK / VW / NT) : (BM * BK / VW / NT);
    constexpr int BV = (BN * BK / VW / NT);
    static_assert(AV >= 1 && BV >= 1, "tile too small");

    // A, k-major: vector i covers row (t + i*NT) / (BK/VW), reduction offset kva
    constexpr int KVPR = BK / VW;               // vectors per k-major row
    constexpr int AVPR = BM / VW;               // vectors per m-major row (A)
    constexpr int BVPR = BN / VW;               // vectors per n-major row (B)

    // precomputed per-row data for gathered rows
    int arow_base[AV];   // FWD: n*H*W*C ; DGRAD: n*P*Q*K ; WGRAD: column m (k-out)
    int arow_h[AV], arow_w[AV];
    bool arow_ok[AV];
    int akv = 0;
    if constexpr (A_KMAJ) {
        akv = (t % KVPR) * VW;
#pragma unroll
        for (int i = 0; i < AV; ++i) {
            long m = m0 + (t + i * NT) / KVPR;
            arow_ok[i] = m < args.M;
            long mm = arow_ok[i] ? m : 0;
            if constexpr (OP == OP_FWD) {
                int q = (int)(mm % g.Q); long tt = mm / g.Q;
                int p = (int)(tt % g.P); int n = (int)(tt / g.P);
                arow_base[i] = n * g.H * g.W * g.C;
                arow_h[i] = p * g.st - g.pad;
                arow_w[i] = q * g.st - g.pad;
                // FAST: a row past M gets a row coordinate that no tap brings
                // into the image, so its range test needs no row mask
                if (FAST && !arow_ok[i]) arow_h[i] = -g.H - g.R;
            } else {  // DGRAD: m = (n, h, w)
                int w = (int)(mm % g.W); long tt = mm / g.W;
                int h = (int)(tt % g.H); int n = (int)(tt / g.H);
                arow_base[i] = n * g.P * g.Q * g.K;
                arow_h[i] = h + g.pad;
                arow_w[i] = w + g.pad;
                if (FAST && !arow_ok[i]) arow_h[i] = -g.P - g.R;
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < AV; ++i) {
            long m = m0 + ((t + i * NT) % AVPR) * VW;
            arow_ok[i] = m < args.M;
            arow_base[i] = (int)m;
            arow_h[i] = arow_w[i] = 0;
        }
    }
    // B
    int bcol_r = 0, bcol_s = 0, bcol_c = 0;
    bool bcol_ok = true;
    bool bcol_ones = false;
    long brow_n[BV];
    bool brow_ok[BV];
    int bkv = 0;
    if constexpr (B_KMAJ) {
        bkv = (t % KVPR) * VW;
#pragma unroll
        for (int i = 0; i < BV; ++i) {
            long n = n0 + (t + i * NT) / KVPR;
            brow_ok[i] = n < args.Ncols;
            brow_n[i] = brow_ok[i] ? n : 0;
        }
    } else {
        long col = n0 + (t % BVPR) * VW;
        bcol_ok = col < args.Ncols;
        if (OP == OP_WGRAD && (args.epi & EPI_BIASCOL) && col == args.Ncols - 1) {
            bcol_ones = true;      // the appended column of ones (bias gradient)
            bcol_ok = false;
        }
        const int cc = bcol_ok ? (int)col : 0;      // below R*S*C < 2^31
        if constexpr (OP == OP_WGRAD) {  // col = (r, s, c)
            if (g.R * g.S == 1) {
                bcol_c = cc;
            } else {
                bcol_c = cc % g.C; const int tt = cc / g.C;
                bcol_s = tt % g.S; bcol_r = tt / g.S;
            }
        } else {                          // DGRAD: col = c
            bcol_c = cc;
        }
#pragma unroll
        for (int i = 0; i < BV; ++i) { brow_n[i] = 0; brow_ok[i] = true; }
    }

    // data gradient: when K is a multiple of the k tile no tile crosses a
    // tap, and row kr of a tile in tap (r, s) at channel c0 reads weight
    // (c0 + kr)*R*S*C + (r*S + s)*C + c: the thread's part is fixed
    // (32-bit with the buffer loads, whose operands are below 2 GB)
    using BOff = std::conditional_t<VW == 4, int, long>;
    const BOff rsc = (BOff)g.R * g.S * g.C;
    const bool dg_one_tap = (OP == OP_DGRAD) && (FAST || g.K % BK == 0);
    BOff b_thr[BV];
#pragma unroll
    for (int i = 0; i < BV; ++i)
        b_thr[i] = (BOff)((t + i * NT) / BVPR) * rsc + bcol_c;

    // two register sets of staged operands (tile kt+2 loads while kt+1 waits
    // to be written to LDS) and their masks; loads are unconditional (masked
    // lanes read the operand's first element) and the mask is applied when
    // the registers are written to LDS
    float areg[2][AV][VW];
    float breg[2][BV][VW];
    bool aok[2][AV], bok[2][BV], bone[2][BV];
    auto ld = [](const float* p, float* v) {
        if constexpr (VW == 4) {
            const float4 t4 = *reinterpret_cast<const float4*>(p);
            v[0] = t4.x; v[1] = t4.y; v[2] = t4.z; v[3] = t4.w;
        } else {
            v[0] = *p;
        }
    };
    // VW = 4: range-checked buffer loads at 32-bit element offsets (every
    // operand below 2 GB, checked by the host), an element off the problem
    // read as zeros through an offset of BUF_OOB, so staging applies no masks
    const long x_el = (long)g.N * g.H * g.W * g.C, dy_el = (long)g.N * g.P * g.Q * g.K;
    const long a_el = (OP == OP_DGRAD) ? dy_el : x_el;
    const long b_el = (OP == OP_WGRAD) ? dy_el : (long)g.K * g.R * g.S * g.C;
    const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(args.a), (short)0, (int)(a_el * 4), BUF_CFG);
    const __amdgpu_buffer_rsrc_t rsb = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(args.b), (short)0, (int)(b_el * 4), BUF_CFG);
    auto ldb = [](__amdgpu_buffer_rsrc_t rs, bool ok, int off, float* v) {
        const uintx4 t = buf_load16(rs, ok ? (unsigned)off * 4u : BUF_OOB, 0u);
        v[0] = __uint_as_float(t[0]); v[1] = __uint_as_float(t[1]);
        v[2] = __uint_as_float(t[2]); v[3] = __uint_as_float(t[3]);
    };

    // The decomposition of the next tile's first reduction index into (filter
    // tap, channel) or (image, output row, output column) is uniform across
    // the workgroup (scalar unit) and stepped from tile to tile (the tiles are
    // staged in order, kt = 0, 1, 2, ...) instead of divided out per tile:
    // FWD / DGRAD tap (nr, ns), its index ntap and the channel offset nc
    // within it; WGRAD the pixel (nn, np, nq).
    int nr = 0, ns = 0, nc = 0, ntap = 0, nq = 0, np = 0, nn = 0;
    const int magS = (256 + g.S - 1) / g.S;   // (t * magS) >> 8 = t / S for t < R*S <= 49
    if constexpr (OP == OP_FWD || OP == OP_DGRAD) {
        if (tap_inner) {
            ntap = tbeg % RSN;
            nc = (tbeg / RSN) * BK;
        } else {
            ntap = (int)kbeg / CCH;
            nc = (int)kbeg - ntap * CCH;
        }
        nr = ntap / g.S;
        ns = ntap - nr * g.S;
    } else {
        nq = (int)kbeg % g.Q;
        const int t0 = (int)kbeg / g.Q;
        np = t0 % g.P;
        nn = t0 / g.P;
    }

    // Staging of one reduction tile [k0, k0 + BK); each thread steps from the
    // tile's decomposition by its own small offset instead of dividing per
    // element.
    auto gload = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        const int T = tbeg + kt;
        // FAST: the loads of the (at most two) tiles past the end read in-range or
        // range-checked offsets and are never staged, so no test is needed
        const bool tin = FAST || T < tend;
        const int k0 = tap_inner ? (tin ? ntap * CCH + nc : 0) : (int)(kbeg + (long)kt * BK);
        // reduction bound of a tile's rows: whole tiles in tap order
        const int kend_i = tap_inner ? (tin ? k0 + BK : 0) : (int)kend;
        if constexpr (OP == OP_FWD || OP == OP_DGRAD) {
            const int CC = CCH;                               // contiguous axis of a tap
            const int c0 = nc, r0 = nr, s0 = ns;
            // the next tile
            if constexpr (FAST) {      // tap index and its (r, s) by a multiply-shift
                ntap = (ntap + 1 == RSN) ? 0 : ntap + 1;
                nc = (ntap == 0) ? nc + BK : nc;
                nr = (ntap * magS) >> 8;
                ns = ntap - nr * g.S;
            } else if (tap_inner) {
                ++ntap;
                if (++ns == g.S) {
                    ns = 0;
                    if (++nr == g.R) { nr = 0; ntap = 0; nc += BK; }
                }
            } else {
                nc += BK;
                while (nc >= CC) { nc -= CC; if (++ns == g.S) { ns = 0; ++nr; } }
            }
            // ---- A: k-major gathered rows ----
            {
                int c = c0 + akv, r = r0, sx = s0;
                if constexpr (!FAST)
                    while (c >= CC) { c -= CC; if (++sx == g.S) { sx = 0; ++r; } }
                const bool kin = FAST ? tin : k0 + akv < kend_i;
#pragma unroll
                for (int i = 0; i < AV; ++i) {
                    if constexpr (OP == OP_FWD) {
                        int h = arow_h[i] + r, w = arow_w[i] + sx;
                        bool ok = (FAST || arow_ok[i]) && kin && (unsigned)h < (unsigned)g.H &&
                                  (unsigned)w < (unsigned)g.W;
                        if constexpr (VW == 4) {
                            ldb(rsa, ok, arow_base[i] + (h * g.W + w) * g.C + c, areg[s][i]);
                        } else {
                            const float* ptr =
                                args.a + (ok ? (arow_base[i] + ((long)h * g.W + w) * g.C + c) : 0);
                            ld(ptr, areg[s][i]);
                        }
                        aok[s][i] = ok;
                    } else {
                        int tp = arow_h[i] - r, tq = arow_w[i] - sx;
                        int p = tp, q = tq;
                        bool ok;
                        if constexpr (FAST) {
                            ok = kin && (unsigned)p < (unsigned)g.P &&
                                 (unsigned)q < (unsigned)g.Q;
                        } else {
                            bool on_grid = true;
                            if (g.st != 1) {        // (uniform branch) strided: exact taps only
                                p = tp / g.st;
                                q = tq / g.st;
                                on_grid = p * g.st == tp && q * g.st == tq;
                            }
                            ok = arow_ok[i] && kin && tp >= 0 && tq >= 0 && on_grid && p < g.P &&
                                 q < g.Q;
                        }
                        if constexpr (VW == 4) {
                            ldb(rsa, ok, arow_base[i] + (p * g.Q + q) * g.K + c, areg[s][i]);
                        } else {
                            const float* ptr =
                                args.a + (ok ? (arow_base[i] + ((long)p * g.Q + q) * g.K + c) : 0);
                            ld(ptr, areg[s][i]);
                        }
                        aok[s][i] = ok;
                    }
                }
            }
            // ---- B ----
#pragma unroll
            for (int i = 0; i < BV; ++i) {
                if constexpr (OP == OP_FWD) {
                    const int kk = k0 + bkv;
                    bool ok = brow_ok[i] && kk < kend_i;
                    if constexpr (VW == 4) {
                        ldb(rsb, ok, (int)brow_n[i] * (int)args.Kred + kk, breg[s][i]);
                    } else {
                        const float* ptr = args.b + (ok ? (brow_n[i] * args.Kred + kk) : 0);
                        ld(ptr, breg[s][i]);
                    }
                    bok[s][i] = ok;
                } else {   // B[kk = (r,s,k)][c] = w[k][r][s][c]
                    const int kr = (t + i * NT) / BVPR;
                    bool ok = bcol_ok && k0 + kr < kend_i;
                    long off;
                    if (dg_one_tap) {
                        // the tile lies within tap (r0, s0): a uniform base plus
                        // this thread's constant offset
                        off = (BOff)c0 * rsc + ((BOff)r0 * g.S + s0) * g.C + b_thr[i];
                    } else {
                        int k = c0 + kr, r = r0, sx = s0;
                        while (k >= CC) { k -= CC; if (++sx == g.S) { sx = 0; ++r; } }
                        off = (((long)k * g.R + r) * g.S + sx) * g.C + bcol_c;
                    }
                    if constexpr (VW == 4) {
                        ldb(rsb, ok, (int)off, breg[s][i]);
                    } else {
                        const float* ptr = args.b + (ok ? off : 0);
                        ld(ptr, breg[s][i]);
                    }
                    bok[s][i] = ok;
                }
            }
        } else {
            // ---- A: dy rows, m-major: A[kk = m'][m = k-out] = dy[m'][k] ----
#pragma unroll
            for (int i = 0; i < AV; ++i) {
                const int kk = k0 + (t + i * NT) / AVPR;
                bool ok = arow_ok[i] && (FAST || kk < kend_i);
                if constexpr (VW == 4) {
                    ldb(rsb, ok, kk * g.K + arow_base[i], areg[s][i]);
                } else {
                    const float* ptr = args.b + (ok ? ((long)kk * g.K + arow_base[i]) : 0);
                    ld(ptr, areg[s][i]);
                }
                aok[s][i] = ok;
            }
            // ---- B: B[kk = (n,p,q)][j = (r,s,c)] = x[n, p*st-pad+r, q*st-pad+s, c] ----
            // (one output pixel per image, as in a fully connected layer: the
            // reduction index is the image)
            const bool px1 = !FAST && g.P * g.Q == 1;
            const int q0 = nq, p0 = np, n0i = nn;
            if constexpr (FAST) {  // the next tile: the next 16 pixels of the row, or the next row
                nq += BK;
                if (nq == g.Q) { nq = 0; if (++np == g.P) { np = 0; ++nn; } }
            } else if (px1) {
                nn += BK;
            } else {
                nq += BK;
                while (nq >= g.Q) { nq -= g.Q; if (++np == g.P) { np = 0; ++nn; } }
            }
#pragma unroll
            for (int i = 0; i < BV; ++i) {
                const int kr = (t + i * NT) / BVPR;
                int q = q0 + kr, p = p0, n = n0i;
                if constexpr (!FAST) {
                    if (px1) {
                        q = 0;
                        n = n0i + kr;
                    } else {
                        while (q >= g.Q) { q -= g.Q; if (++p == g.P) { p = 0; ++n; } }
                    }
                }
                const bool kin = FAST || k0 + kr < kend_i;
                int h = p * g.st - g.pad + bcol_r, w = q * g.st - g.pad + bcol_s;
                bool ok = bcol_ok && kin && (unsigned)h < (unsigned)g.H &&
                          (unsigned)w < (unsigned)g.W;
                if constexpr (VW == 4) {
                    ldb(rsa, ok, ((n * g.H + h) * g.W + w) * g.C + bcol_c, breg[s][i]);
                } else {
                    const float* ptr =
                        args.a + (ok ? ((((long)n * g.H + h) * g.W + w) * g.C + bcol_c) : 0);
                    ld(ptr, breg[s][i]);
                }
                bok[s][i] = ok;
                bone[s][i] = bcol_ones && kin;
            }
        }
    };

    auto sstore = [&](auto S) {
        constexpr int s = decltype(S)::value;
        float* As = smem + s * BK * (LDA + LDB);
        float* Bs = As + BK * LDA;
#pragma unroll
        for (int i = 0; i < AV; ++i) {
            if constexpr (A_KMAJ) {
                int row = (t + i * NT) / KVPR;
#pragma unroll
                for (int j = 0; j < VW; ++j)
                    As[(akv + j) * LDA + row] = (VW == 4 || aok[s][i]) ? areg[s][i][j] : 0.f;
            } else {
                int kr = (t + i * NT) / AVPR;
                int col = ((t + i * NT) % AVPR) * VW;
#pragma unroll
                for (int j = 0; j < VW; ++j)
                    As[kr * LDA + col + j] = (VW == 4 || aok[s][i]) ? areg[s][i][j] : 0.f;
            }
        }
#pragma unroll
        for (int i = 0; i < BV; ++i) {
            if constexpr (B_KMAJ) {
                int row = (t + i * NT) / KVPR;
#pragma unroll
                for (int j = 0; j < VW; ++j)
                    Bs[(bkv + j) * LDB + row] = (VW == 4 || bok[s][i]) ? breg[s][i][j] : 0.f;
            } else {
                int kr = (t + i * NT) / BVPR;
                int col = ((t + i * NT) % BVPR) * VW;
#pragma unroll
                for (int j = 0; j < VW; ++j) {
                    // the appended column of ones (bias gradient) in lane 0
                    // (VW = 4: an element off the problem was read as zero, and
                    // the ones column, weight gradient only, is read past the end)
                    const bool ones = OP == OP_WGRAD && bone[s][i];
                    const float one = (j == 0 && ones) ? 1.f : 0.f;
                    Bs[kr * LDB + col + j] = (VW == 4) ? (ones ? one : breg[s][i][j])
                                                       : (bok[s][i] ? breg[s][i][j] : one);
                }
            }
        }
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int lr = lane & 31;
    const int lk = lane >> 5;
    // one k tile: prefetch tile kt+2 into register set s, multiply LDS buffer
    // s, write tile kt+1 (register set s^1) to LDS buffer s^1; loads of tiles
    // past the end are fully masked, so every load is on one path and the
    // wait before the LDS write counts only the older set.  The wave raises
    // its issue priority while it multiplies, so that of the waves sharing a
    // SIMD the ones with MFMAs ready go ahead of those staging operands (the
    // kernels below do the same).
    auto step = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        gload(kt + 2, S);
        const float* As = smem + s * BK * (LDA + LDB);
        const float* Bs = As + BK * LDA;
        __builtin_amdgcn_s_setprio(1);
        if (kt < ktiles) {
#pragma unroll
            for (int kk = 0; kk < BK; kk += 2) {
                const float* ar = As + (kk + lk) * LDA + wm + lr;
                const float* br = Bs + (kk + lk) * LDB + wn + lr;
                float av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) av[i] = ar[32 * i];
#pragma unroll
                for (int j = 0; j < TN; ++j) bv[j] = br[32 * j];
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j],
                                                                        0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        if (kt + 1 < ktiles) sstore(std::integral_constant<int, s ^ 1>{});
        __syncthreads();
    };

    const std::integral_constant<int, 0> I0{};
    const std::integral_constant<int, 1> I1{};
    gload(0, I0);
    gload(1, I1);
    if (ktiles > 0) sstore(I0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; kt += 2) {
        step(kt, I0);
        step(kt + 1, I1);
    }

    static_assert(sizeof(smem) >= (NT / 64) * SLOT_FLOATS * sizeof(float), "epilogue slots");
    write_tile<BM, BN, TM, TN, WIDE>(args, wk, acc, wm, wn, lane,
                                     reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS,
                                     reinterpret_cast<float*>(smem));
}

// ---- fp32 weight gradient of a fully connected layer -------------------------
// dW[m][n] = sum_k dy[k][m] x[k][n], the reduction over a batch of at most 32
// images: a rank-k update that writes far more than it computes (4 bytes per
// output against 2k flops), so the order of its writes sets its speed.  A
// fixed grid of workgroups walks the FCW_BM x FCW_BN tiles in row-major order
// (workgroup w takes tiles w, w + G, w + 2G, ... of G workgroups), so the
// tiles being written at any time form one contiguous run of whole output
// rows.  Each tile stages its dy and x rows (both read from L2) through LDS,
// the next tile's loads in flight while the current one is multiplied and
// written.  Four waves of 64 x 64 (2 x 2 MFMA 32x32x2 tiles); rows k past the
// batch are zeros.  The epilogue is a plain store (no bias, activation, mask
// or accumulation applies to a weight gradient).  The bias gradient (the sum
// of dy over the batch, in batch order) is written with the first tile of
// each row block.
constexpr int FCW_BM = 64, FCW_BN = 256, FCW_KMAX = 32;
constexpr int FCW_LDA = FCW_BM + PAD_V, FCW_LDB = FCW_BN + PAD_V;

__global__ void __launch_bounds__(256, 2) fcw_kernel(KArgs args) {
    static_assert((FCW_BM / 64) * (FCW_BN / 64) == 4, "four waves of 64 x 64");
    __shared__ float sA[FCW_KMAX * FCW_LDA];
    __shared__ float sB[FCW_KMAX * FCW_LDB];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    constexpr int WAVES_N = FCW_BN / 64;
    const int wm = (wave / WAVES_N) * 64, wn = (wave % WAVES_N) * 64;
    const int bias = (args.epi & EPI_BIASCOL) ? 1 : 0;
    const int M = (int)args.M, Nw = (int)args.Ncols - bias, K = (int)args.Kred;
    const int tiles_n = (Nw + FCW_BN - 1) / FCW_BN;
    const int tiles = args.tiles_m * tiles_n;
    const float* dy = args.b;          // [K][M]
    const float* x = args.a;           // [K][Nw]
    // staging: thread t holds 4 columns of rows t / (B/4) + (1024/B) i
    constexpr int AT = FCW_BM / 4, AR = 256 / AT, AV = FCW_KMAX / AR;
    constexpr int BT = FCW_BN / 4, BR = 256 / BT, BV = FCW_KMAX / BR;
    float4 na[AV], nb[BV];
    auto load = [&](int T) {
        const int m0 = (T / tiles_n) * FCW_BM, n0 = (T % tiles_n) * FCW_BN;
#pragma unroll
        for (int i = 0; i < AV; ++i) {
            const int k = t / AT + AR * i, m = m0 + (t % AT) * 4;
            na[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (k < K && m < M) na[i] = *reinterpret_cast<const float4*>(dy + (long)k * M + m);
        }
#pragma unroll
        for (int i = 0; i < BV; ++i) {
            const int k = t / BT + BR * i, n = n0 + (t % BT) * 4;
            nb[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (k < K && n < Nw) nb[i] = *reinterpret_cast<const float4*>(x + (long)k * Nw + n);
        }
    };
    const int lr = lane & 31, lk = lane >> 5;
    const int kp = (K + 1) & ~1;
    if ((int)blockIdx.x < tiles) load(blockIdx.x);
    for (int T = blockIdx.x; T < tiles; T += gridDim.x) {
        const int mt = T / tiles_n, nt = T - mt * tiles_n;
#pragma unroll
        for (int i = 0; i < AV; ++i)
            *reinterpret_cast<float4*>(sA + (t / AT + AR * i) * FCW_LDA + (t % AT) * 4) = na[i];
#pragma unroll
        for (int i = 0; i < BV; ++i)
            *reinterpret_cast<float4*>(sB + (t / BT + BR * i) * FCW_LDB + (t % BT) * 4) = nb[i];
        __syncthreads();
        if (T + (int)gridDim.x < tiles) load(T + gridDim.x);
        if (bias && nt == 0 && t < FCW_BM && mt * FCW_BM + t < M) {
            float s = 0.f;
            for (int k = 0; k < K; ++k) s += sA[k * FCW_LDA + t];
            args.bias_out[mt * FCW_BM + t] = s;
        }
        floatx16 acc[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
        for (int kk = 0; kk < kp; kk += 2) {
            const float* ar = sA + (kk + lk) * FCW_LDA + wm + lr;
            const float* br = sB + (kk + lk) * FCW_LDB + wn + lr;
            const float av[2] = {ar[0], ar[32]}, bv[2] = {br[0], br[32]};
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0,
                                                                    0);
        }
        __syncthreads();               // sA, sB free for the next tile
        // the tile straight from the accumulators: a store writes 32
        // consecutive columns (128 bytes) of two rows
        const int r0 = mt * FCW_BM + wm + 4 * lk;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int col = nt * FCW_BN + wn + 32 * j + lr;
            if (col >= Nw) continue;
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = r0 + 32 * i + 8 * (v >> 2) + (v & 3);
                    if (row < M) args.out[(long)row * Nw + col] = acc[i][j][v];
                }
        }
    }
}

// ---- fp32 forward of a fully connected layer ----------------------------------
// y[m][n] = sum_k x[m][k] w[n][k] over at most 32 images: the layer streams
// its weights (4 bytes each) for 2M flops per weight, so how the weight rows
// are read sets its speed.  A workgroup owns FCF_BN output columns and one
// chunk of the reduction; its four waves take each 128-wide k step of the
// chunk in four 32-wide parts, so a step reads its weight rows in 512-byte
// runs.  No LDS staging: a lane loads 16-byte pieces of one x row and of two
// weight rows straight into MFMA operand registers.  The 32x32x2 MFMA's two k
// slots are taken as the two lane halves' 16-element runs and its sixteen
// issues as the elements of the runs, for both operands alike, which leaves
// the sum unchanged.  The waves' sums are added in LDS in wave order and
// written as the chunk's partial tile (32 x FCF_BN); the cut-tile reduction
// adds the chunks in order and applies bias and ReLU.
constexpr int FCF_BN = 64, FCF_KW = 32, FCF_KSTEP = 4 * FCF_KW, FCF_NS = 2;

__global__ void __launch_bounds__(256, 2) fcf_kernel(KArgs args) {
    __shared__ float red[4][2][16][64];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int lr = lane & 31, lh = lane >> 5;
    const int nt = blockIdx.x % args.tiles_n, z = blockIdx.x / args.tiles_n;
    const int M = (int)args.M, N = (int)args.Ncols, K = (int)args.Kred;
    const int kbeg = z * args.kchunk, kend = min(kbeg + args.kchunk, K);
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(args.a), (short)0, M * K * 4, BUF_CFG);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(args.b), (short)0, N * K * 4, BUF_CFG);
    const int n0 = nt * FCF_BN;
    const bool mok = lr < M, nok0 = n0 + lr < N, nok1 = n0 + 32 + lr < N;
    const unsigned xrow = (unsigned)(lr * K), w0 = (unsigned)((n0 + lr) * K);
    const unsigned w1 = (unsigned)((n0 + 32 + lr) * K);
    floatx16 acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
    // FCF_NS register stages: the loads of the wave's next FCF_NS - 1 parts
    // are in flight while one part is multiplied
    uintx4 xa[FCF_NS][4], wa[FCF_NS][2][4];
    auto load = [&](int s, int k0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = k0 + 16 * lh + 4 * q;
            const bool kin = k < kend;
            xa[s][q] = buf_load16(rx, (mok && kin) ? (xrow + k) * 4u : BUF_OOB, 0u);
            wa[s][0][q] = buf_load16(rw, (nok0 && kin) ? (w0 + k) * 4u : BUF_OOB, 0u);
            wa[s][1][q] = buf_load16(rw, (nok1 && kin) ? (w1 + k) * 4u : BUF_OOB, 0u);
        }
    };
    auto mma = [&](int s) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                        __uint_as_float(xa[s][q][e]), __uint_as_float(wa[s][j][q][e]), acc[j], 0,
                        0, 0);
    };
    const int kq = kbeg + FCF_KW * wave;     // the wave's first part
#pragma unroll
    for (int s = 0; s < FCF_NS - 1; ++s)
        if (kq + s * FCF_KSTEP < kend) load(s, kq + s * FCF_KSTEP);
    for (int base = kq; base < kend; base += FCF_NS * FCF_KSTEP) {
#pragma unroll
        for (int s = 0; s < FCF_NS; ++s) {
            const int k = base + s * FCF_KSTEP;
            if (k < kend) {
                const int kn = k + (FCF_NS - 1) * FCF_KSTEP;
                if (kn < kend) load((s + FCF_NS - 1) % FCF_NS, kn);
                mma(s);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[wave][j][v][lane] = acc[j][v];
    __syncthreads();
    if (wave < 2) {
        const int j = wave;
        float* dst = args.ws + ((long)nt * args.splits + z) * (32 * FCF_BN);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const float s = ((red[0][j][v][lane] + red[1][j][v][lane]) + red[2][j][v][lane]) +
                            red[3][j][v][lane];
            dst[(8 * (v >> 2) + 4 * lh + (v & 3)) * FCF_BN + 32 * j + lr] = s;
        }
    }
}

// ---- bf16 kernel ------------------------------------------------------------
// The same three contractions on v_mfma_f32_32x32x16_bf16.  Operands are
// gathered in fp32 exactly as above, rounded to bf16 and staged row-major in
// LDS with the reduction index contiguous: [rows][LDH] bf16, BKH = 32 k per
// tile, rows padded to 80 bytes so that the 16-byte fragment reads of 8
// consecutive rows cover all banks once.  A lane's MFMA operand is 8
// consecutive k of one row (row = lane % 32, k = 8 (lane / 32) .. + 7; both
// operands use the same k order, so the contraction is the same whatever
// order the hardware takes the k in).
//
// k-major operands (gathered rows, reduction index contiguous in memory) are
// staged in groups of 4 consecutive k of one row (one 8-byte LDS store);
// m-major operands (reduction index = memory row) in 4 x 4 blocks, 4
// reduction rows of 4 consecutive columns, transposed in registers.
constexpr int BKH = 32;
constexpr int LDH = BKH + 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned uintx2 __attribute__((ext_vector_type(2)));

template <int OP, int BM, int BN, int WM, int WN, int VW>
__global__ void __launch_bounds__(64 * (BM / WM) * (BN / WN), 2) igemm_bf16_kernel(KArgs args) {
    constexpr int NT = 64 * (BM / WM) * (BN / WN);
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr bool A_KMAJ = (OP != OP_WGRAD);
    constexpr bool B_KMAJ = (OP == OP_FWD);
    constexpr int WAVES_N = BN / WN;
    constexpr int KG = BKH / 4;                  // 4-k groups per k-major row
    constexpr int GA = BM * KG / NT;             // k-major groups per thread
    constexpr int GB = BN * KG / NT;
    constexpr int CGA = BM / 4, CGB = BN / 4;    // column groups of an m-major operand
    constexpr int PA = (2 * BM + NT - 1) / NT;   // m-major 4x4 blocks per thread
    constexpr int PB = (2 * BN + NT - 1) / NT;
    constexpr int NA = A_KMAJ ? GA : 4 * PA;     // 4-vectors held per thread
    constexpr int NB = B_KMAJ ? GB : 4 * PB;
    constexpr int CV = VW == 4 ? 1 : 4;          // separately addressed columns of a 4-vector
    static_assert(GA >= 1 && GB >= 1 && NT % KG == 0 && NT % CGA == 0 && NT % CGB == 0,
                  "tile shape");
    __shared__ __attribute__((aligned(16))) unsigned short smem[2 * (BM + BN) * LDH];

    const ConvGeo& g = args.g;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int wm = (wave / WAVES_N) * WM;
    const int wn = (wave % WAVES_N) * WN;
    const Work wk = decode_work<BM, BN>(args);
    const int ktiles = (int)((wk.kend - wk.kbeg + BKH - 1) / BKH);
    const int kg = (t % KG) * 4;                                // k-major: k offset of the group
    const bool a_act = A_KMAJ || 2 * BM >= NT || t < 2 * BM;    // m-major: thread owns a block
    const bool b_act = B_KMAJ || 2 * BN >= NT || t < 2 * BN;

    // ---- per-thread staging coordinates ----
    int arow_base[GA], arow_h[GA], arow_w[GA];
    bool arow_ok[GA];
    long acol = 0;
    if constexpr (A_KMAJ) {
#pragma unroll
        for (int i = 0; i < GA; ++i) {
            const long m = wk.m0 + t / KG + i * (NT / KG);
            arow_ok[i] = m < args.M;
            const long mm = arow_ok[i] ? m : 0;
            if constexpr (OP == OP_FWD) {
                int q = (int)(mm % g.Q); long tt = mm / g.Q;
                int p = (int)(tt % g.P); int n = (int)(tt / g.P);
                arow_base[i] = n * g.H * g.W * g.C;
                arow_h[i] = p * g.st - g.pad;
                arow_w[i] = q * g.st - g.pad;
            } else {  // DGRAD: m = (n, h, w)
                int w = (int)(mm % g.W); long tt = mm / g.W;
                int h = (int)(tt % g.H); int n = (int)(tt / g.H);
                arow_base[i] = n * g.P * g.Q * g.K;
                arow_h[i] = h + g.pad;
                arow_w[i] = w + g.pad;
            }
        }
    } else {
        acol = wk.m0 + (t % CGA) * 4;           // WGRAD: output channels acol .. +3
    }
    long brow_n[GB];
    bool brow_ok[GB];
    long bcol = 0;
    int bcol_r[CV], bcol_s[CV], bcol_c[CV];
    bool bcol_ok[CV], bcol_ones[CV];
    if constexpr (B_KMAJ) {
#pragma unroll
        for (int i = 0; i < GB; ++i) {
            const long n = wk.n0 + t / KG + i * (NT / KG);
            brow_ok[i] = n < args.Ncols;
            brow_n[i] = brow_ok[i] ? n : 0;
        }
    } else {
        bcol = wk.n0 + (t % CGB) * 4;
#pragma unroll
        for (int c = 0; c < CV; ++c) {
            const long col = bcol + c;
            bcol_ok[c] = col < args.Ncols;
            bcol_ones[c] = false;
            if (OP == OP_WGRAD && (args.epi & EPI_BIASCOL) && col == args.Ncols - 1) {
                bcol_ones[c] = true;       // the appended column of ones (bias gradient)
                bcol_ok[c] = false;
            }
            const long cc = bcol_ok[c] ? col : 0;
            if constexpr (OP == OP_WGRAD) {      // col = (r, s, c)
                bcol_c[c] = (int)(cc % g.C); long tt = cc / g.C;
                bcol_s[c] = (int)(tt % g.S); bcol_r[c] = (int)(tt / g.S);
            } else {                              // DGRAD: col = c
                bcol_c[c] = (int)cc;
                bcol_r[c] = bcol_s[c] = 0;
            }
        }
    }

    float areg[NA][4];
    float breg[NB][4];

    // Staging of one reduction tile [k0, k0 + BKH); as in the fp32 kernel the
    // decomposition of k0 is uniform and each thread steps from it.
    auto gload = [&](int kt) {
        const int k0 = (int)(wk.kbeg + (long)kt * BKH);
        const int kend_i = (int)wk.kend;
        if constexpr (OP == OP_FWD || OP == OP_DGRAD) {
            const int CC = (OP == OP_FWD) ? g.C : g.K;       // contiguous axis of a tap
            const int rs0 = k0 / CC;
            const int c0 = k0 - rs0 * CC;
            const int r0 = rs0 / g.S;
            const int s0 = rs0 - r0 * g.S;
            // ---- A: k-major gathered rows, k = k0 + kg .. + 3 ----
            {
                int c = c0 + kg, r = r0, sx = s0;
                while (c >= CC) { c -= CC; if (++sx == g.S) { sx = 0; ++r; } }
#pragma unroll
                for (int j = 0; j < CV; ++j) {
                    if (j > 0 && ++c == CC) { c = 0; if (++sx == g.S) { sx = 0; ++r; } }
                    const bool kin = k0 + kg + j < kend_i;
#pragma unroll
                    for (int i = 0; i < GA; ++i) {
                        bool ok;
                        long off;
                        if constexpr (OP == OP_FWD) {
                            const int h = arow_h[i] + r, w = arow_w[i] + sx;
                            ok = arow_ok[i] && kin && (unsigned)h < (unsigned)g.H &&
                                 (unsigned)w < (unsigned)g.W;
                            off = arow_base[i] + ((long)h * g.W + w) * g.C + c;
                        } else {
                            const int tp = arow_h[i] - r, tq = arow_w[i] - sx;
                            int p = tp, q = tq;
                            bool on_grid = true;
                            if (g.st != 1) {        // (uniform branch) strided: exact taps only
                                p = tp / g.st;
                                q = tq / g.st;
                                on_grid = p * g.st == tp && q * g.st == tq;
                            }
                            ok = arow_ok[i] && kin && tp >= 0 && tq >= 0 && on_grid &&
                                 p < g.P && q < g.Q;
                            off = arow_base[i] + ((long)p * g.Q + q) * g.K + c;
                        }
                        const float* ptr = args.a + (ok ? off : 0);
                        if constexpr (VW == 4) load_vec<4>(ptr, ok, areg[i]);
                        else areg[i][j] = ok ? *ptr : 0.f;
                    }
                }
            }
            // ---- B ----
            if constexpr (OP == OP_FWD) {                     // weight rows, k-major
#pragma unroll
                for (int j = 0; j < CV; ++j) {
                    const int kk = k0 + kg + j;
#pragma unroll
                    for (int i = 0; i < GB; ++i) {
                        const bool ok = brow_ok[i] && kk < kend_i;
                        const float* ptr = args.b + (ok ? (brow_n[i] * args.Kred + kk) : 0);
                        if constexpr (VW == 4) load_vec<4>(ptr, ok, breg[i]);
                        else breg[i][j] = ok ? *ptr : 0.f;
                    }
                }
            } else if (b_act) {     // B[kk = (r,s,k)][c] = w[k][r][s][c], m-major blocks
#pragma unroll
                for (int i = 0; i < PB; ++i) {
                    const int kq = ((t + i * NT) / CGB) * 4;
                    int k = c0 + kq, r = r0, sx = s0;
                    while (k >= CC) { k -= CC; if (++sx == g.S) { sx = 0; ++r; } }
#pragma unroll
                    for (int jr = 0; jr < 4; ++jr) {
                        if (jr > 0 && ++k == CC) { k = 0; if (++sx == g.S) { sx = 0; ++r; } }
                        const bool kin = k0 + kq + jr < kend_i;
                        const long base = (((long)k * g.R + r) * g.S + sx) * g.C;
#pragma unroll
                        for (int c = 0; c < CV; ++c) {
                            const bool ok = bcol_ok[c] && kin;
                            const float* ptr = args.b + (ok ? base + bcol_c[c] : 0);
                            if constexpr (VW == 4) load_vec<4>(ptr, ok, breg[4 * i + jr]);
                            else breg[4 * i + jr][c] = ok ? *ptr : 0.f;
                        }
                    }
                }
            }
        } else {
            // ---- A: A[kk = m'][m = k-out] = dy[m'][k], m-major blocks ----
            if (a_act) {
#pragma unroll
                for (int i = 0; i < PA; ++i) {
                    const int kq = ((t + i * NT) / CGA) * 4;
#pragma unroll
                    for (int jr = 0; jr < 4; ++jr) {
                        const int kk = k0 + kq + jr;
                        const bool kin = kk < kend_i;
                        const float* row = args.b + (long)kk * g.K + acol;
                        if constexpr (VW == 4) {
                            const bool ok = kin && acol < args.M;
                            load_vec<4>(ok ? row : args.b, ok, areg[4 * i + jr]);
                        } else {
#pragma unroll
                            for (int c = 0; c < 4; ++c) {
                                const bool ok = kin && acol + c < args.M;
                                areg[4 * i + jr][c] = ok ? row[c] : 0.f;
                            }
                        }
                    }
                }
            }
            // ---- B: B[kk = (n,p,q)][j = (r,s,c)] = x[n, p*st-pad+r, q*st-pad+s, c] ----
            if (b_act) {
                const int q0 = k0 % g.Q;
                const int t0 = k0 / g.Q;
                const int p0 = t0 % g.P;
                const int n0i = t0 / g.P;
#pragma unroll
                for (int i = 0; i < PB; ++i) {
                    const int kq = ((t + i * NT) / CGB) * 4;
                    int q = q0 + kq, p = p0, n = n0i;
                    while (q >= g.Q) { q -= g.Q; if (++p == g.P) { p = 0; ++n; } }
#pragma unroll
                    for (int jr = 0; jr < 4; ++jr) {
                        if (jr > 0 && ++q == g.Q) { q = 0; if (++p == g.P) { p = 0; ++n; } }
                        const bool kin = k0 + kq + jr < kend_i;
#pragma unroll
                        for (int c = 0; c < CV; ++c) {
                            const int h = p * g.st - g.pad + bcol_r[c];
                            const int w = q * g.st - g.pad + bcol_s[c];
                            const bool ok = bcol_ok[c] && kin && (unsigned)h < (unsigned)g.H &&
                                            (unsigned)w < (unsigned)g.W;
                            const float* ptr =
                                args.a +
                                (ok ? ((((long)n * g.H + h) * g.W + w) * g.C + bcol_c[c]) : 0);
                            if constexpr (VW == 4) {
                                load_vec<4>(ptr, ok, breg[4 * i + jr]);
                                if (bcol_ones[0]) {
                                    breg[4 * i + jr][0] = kin ? 1.f : 0.f;
                                    breg[4 * i + jr][1] = breg[4 * i + jr][2] =
                                        breg[4 * i + jr][3] = 0.f;
                                }
                            } else {
                                breg[4 * i + jr][c] =
                                    bcol_ones[c] ? (kin ? 1.f : 0.f) : (ok ? *ptr : 0.f);
                            }
                        }
                    }
                }
            }
        }
    };

    auto sstore = [&](int buf) {
        unsigned short* As = smem + buf * (BM + BN) * LDH;
        unsigned short* Bs = As + BM * LDH;
        if constexpr (A_KMAJ) {
#pragma unroll
            for (int i = 0; i < GA; ++i) {
                const int row = t / KG + i * (NT / KG);
                *reinterpret_cast<uintx2*>(As + row * LDH + kg) =
                    uintx2{pack_bf16(areg[i][0], areg[i][1]), pack_bf16(areg[i][2], areg[i][3])};
            }
        } else if (a_act) {
#pragma unroll
            for (int i = 0; i < PA; ++i) {
                const int kq = ((t + i * NT) / CGA) * 4;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int col = (t % CGA) * 4 + c;
                    *reinterpret_cast<uintx2*>(As + col * LDH + kq) =
                        uintx2{pack_bf16(areg[4 * i][c], areg[4 * i + 1][c]),
                               pack_bf16(areg[4 * i + 2][c], areg[4 * i + 3][c])};
                }
            }
        }
        if constexpr (B_KMAJ) {
#pragma unroll
            for (int i = 0; i < GB; ++i) {
                const int row = t / KG + i * (NT / KG);
                *reinterpret_cast<uintx2*>(Bs + row * LDH + kg) =
                    uintx2{pack_bf16(breg[i][0], breg[i][1]), pack_bf16(breg[i][2], breg[i][3])};
            }
        } else if (b_act) {
#pragma unroll
            for (int i = 0; i < PB; ++i) {
                const int kq = ((t + i * NT) / CGB) * 4;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int col = (t % CGB) * 4 + c;
                    *reinterpret_cast<uintx2*>(Bs + col * LDH + kq) =
                        uintx2{pack_bf16(breg[4 * i][c], breg[4 * i + 1][c]),
                               pack_bf16(breg[4 * i + 2][c], breg[4 * i + 3][c])};
                }
            }
        }
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    if (ktiles > 0) {
        gload(0);
        sstore(0);
    }
    __syncthreads();
    const int lr = lane & 31;
    const int lk = lane >> 5;
    for (int kt = 0; kt < ktiles; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < ktiles) gload(kt + 1);
        const unsigned short* As = smem + buf * (BM + BN) * LDH;
        const unsigned short* Bs = As + BM * LDH;
#pragma unroll
        for (int kk = 0; kk < BKH; kk += 16) {
            bf16x8 av[TM], bv[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                av[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(
                                                       As + (wm + 32 * i + lr) * LDH + kk + 8 * lk));
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bv[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(
                                                       Bs + (wn + 32 * j + lr) * LDH + kk + 8 * lk));
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0,
                                                                         0, 0);
        }
        if (kt + 1 < ktiles) sstore(buf ^ 1);
        __syncthreads();
    }
    static_assert(sizeof(smem) >= (NT / 64) * SLOT_FLOATS * sizeof(float), "epilogue slots");
    write_tile<BM, BN, TM, TN>(args, wk, acc, wm, wn, lane,
                               reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS,
                               reinterpret_cast<float*>(smem));
}


// ---- bf16 kernel on bf16 operands -------------------------------------------
// The bf16 contractions when both operands are already rounded to bf16 in
// memory (a16 / b16), on the same MFMA and the same LDS row layout as
// igemm_bf16_kernel, with BKX k per tile (rows padded by 8 bf16, so 16-byte
// fragment reads of 8 consecutive rows still cover all banks once).  k-major
// operands load 8 consecutive k (16 bytes) of a row and store them with one
// 16-byte LDS write; m-major operands load 4 x 4 blocks (4 reduction rows of
// 4 columns, 8 bytes each) and transpose them in registers.
//
// Staging runs two tiles ahead: while the MFMAs consume tile kt from LDS,
// the loads of tile kt+2 are in flight into one register set and tile kt+1,
// loaded one step earlier into the other set, is written to the second LDS
// buffer.  Every load is issued unconditionally (masked lanes read the
// operand's first element) and the mask is applied when the registers are
// written to LDS, so the wait before that write covers only the older loads.
// Used only when every contiguous axis is a multiple of 8 elements and the
// operands are 16-byte aligned, so there is no scalar path and no bias column.
template <int OP, int BM, int BN, int WM, int WN, int BKX>
__global__ void __launch_bounds__(64 * (BM / WM) * (BN / WN), 2) igemm_h16_kernel(KArgs args) {
    constexpr int NT = 64 * (BM / WM) * (BN / WN);
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int LDX = BKX + 8;
    constexpr bool A_KMAJ = (OP != OP_WGRAD);
    constexpr bool B_KMAJ = (OP == OP_FWD);
    constexpr int WAVES_N = BN / WN;
    constexpr int KG = BKX / 8;                  // 8-k groups per k-major row
    constexpr int GA = BM * KG / NT;             // k-major groups per thread
    constexpr int GB = BN * KG / NT;
    constexpr int CGA = BM / 4, CGB = BN / 4;    // column groups of an m-major operand
    constexpr int NBA = (BKX / 4) * CGA;         // 4x4 blocks of an m-major tile
    constexpr int NBB = (BKX / 4) * CGB;
    constexpr int PA = (NBA + NT - 1) / NT;      // m-major blocks per thread
    constexpr int PB = (NBB + NT - 1) / NT;
    static_assert(BKX % 16 == 0 && GA >= 1 && GB >= 1 && NT % KG == 0 &&
                  (BM * KG) % NT == 0 && (BN * KG) % NT == 0 && NT % CGA == 0 &&
                  NT % CGB == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) unsigned short smem[2 * (BM + BN) * LDX];

    const ConvGeo& g = args.g;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int wm = (wave / WAVES_N) * WM;
    const int wn = (wave % WAVES_N) * WN;
    const Work wk = decode_work<BM, BN>(args);
    const int ktiles = (int)((wk.kend - wk.kbeg + BKX - 1) / BKX);
    const int kg = (t % KG) * 8;
    const unsigned short* A = args.a16;
    const unsigned short* Bm = args.b16;

    int arow_base[GA], arow_h[GA], arow_w[GA];
    bool arow_ok[GA];
    long acol = 0;
    if constexpr (A_KMAJ) {
#pragma unroll
        for (int i = 0; i < GA; ++i) {
            const long m = wk.m0 + t / KG + i * (NT / KG);
            arow_ok[i] = m < args.M;
            const long mm = arow_ok[i] ? m : 0;
            if constexpr (OP == OP_FWD) {
                int q = (int)(mm % g.Q); long tt = mm / g.Q;
                int p = (int)(tt % g.P); int n = (int)(tt / g.P);
                arow_base[i] = n * g.H * g.W * g.C;
                arow_h[i] = p * g.st - g.pad;
                arow_w[i] = q * g.st - g.pad;
            } else {
                int w = (int)(mm % g.W); long tt = mm / g.W;
                int h = (int)(tt % g.H); int n = (int)(tt / g.H);
                arow_base[i] = n * g.P * g.Q * g.K;
                arow_h[i] = h + g.pad;
                arow_w[i] = w + g.pad;
            }
        }
    } else {
        acol = wk.m0 + (t % CGA) * 4;
    }
    long brow_n[GB];
    bool brow_ok[GB];
    long bcol = 0;
    int bcol_r = 0, bcol_s = 0, bcol_c = 0;
    bool bcol_ok = false;
    if constexpr (B_KMAJ) {
#pragma unroll
        for (int i = 0; i < GB; ++i) {
            const long n = wk.n0 + t / KG + i * (NT / KG);
            brow_ok[i] = n < args.Ncols;
            brow_n[i] = brow_ok[i] ? n : 0;
        }
    } else {
        bcol = wk.n0 + (t % CGB) * 4;
        bcol_ok = bcol < args.Ncols;
        const long cc = bcol_ok ? bcol : 0;
        if constexpr (OP == OP_WGRAD) {
            bcol_c = (int)(cc % g.C); long tt = cc / g.C;
            bcol_s = (int)(tt % g.S); bcol_r = (int)(tt / g.S);
        } else {
            bcol_c = (int)cc;
        }
    }

    // two register sets of staged operands and their masks
    uintx4 ra_k[2][A_KMAJ ? GA : 1], rb_k[2][B_KMAJ ? GB : 1];
    uintx2 ra_m[2][A_KMAJ ? 1 : 4 * PA], rb_m[2][B_KMAJ ? 1 : 4 * PB];
    bool ma_k[2][A_KMAJ ? GA : 1], mb_k[2][B_KMAJ ? GB : 1];
    bool ma_m[2][A_KMAJ ? 1 : 4 * PA], mb_m[2][B_KMAJ ? 1 : 4 * PB];

    auto ld16 = [](const unsigned short* p) -> uintx4 {
        return *reinterpret_cast<const uintx4*>(p);
    };
    auto ld8 = [](const unsigned short* p) -> uintx2 {
        return *reinterpret_cast<const uintx2*>(p);
    };

    auto gload = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        const int k0 = (int)(wk.kbeg + (long)kt * BKX);
        const int kend_i = (int)wk.kend;
        if constexpr (OP == OP_FWD || OP == OP_DGRAD) {
            const int CC = (OP == OP_FWD) ? g.C : g.K;
            const int rs0 = k0 / CC;
            const int c0 = k0 - rs0 * CC;
            const int r0 = rs0 / g.S;
            const int s0 = rs0 - r0 * g.S;
            {
                int c = c0 + kg, r = r0, sx = s0;
                while (c >= CC) { c -= CC; if (++sx == g.S) { sx = 0; ++r; } }
                const bool kin = k0 + kg < kend_i;
#pragma unroll
                for (int i = 0; i < GA; ++i) {
                    bool ok;
                    long off;
                    if constexpr (OP == OP_FWD) {
                        const int h = arow_h[i] + r, w = arow_w[i] + sx;
                        ok = arow_ok[i] && kin && (unsigned)h < (unsigned)g.H &&
                             (unsigned)w < (unsigned)g.W;
                        off = arow_base[i] + ((long)h * g.W + w) * g.C + c;
                    } else {
                        const int tp = arow_h[i] - r, tq = arow_w[i] - sx;
                        int p = tp, q = tq;
                        bool on_grid = true;
                        if (g.st != 1) {
                            p = tp / g.st;
                            q = tq / g.st;
                            on_grid = p * g.st == tp && q * g.st == tq;
                        }
                        ok = arow_ok[i] && kin && tp >= 0 && tq >= 0 && on_grid && p < g.P &&
                             q < g.Q;
                        off = arow_base[i] + ((long)p * g.Q + q) * g.K + c;
                    }
                    ra_k[s][i] = ld16(A + (ok ? off : 0));
                    ma_k[s][i] = ok;
                }
            }
            if constexpr (OP == OP_FWD) {
                const int kk = k0 + kg;
#pragma unroll
                for (int i = 0; i < GB; ++i) {
                    const bool ok = brow_ok[i] && kk < kend_i;
                    rb_k[s][i] = ld16(Bm + (ok ? (brow_n[i] * args.Kred + kk) : 0));
                    mb_k[s][i] = ok;
                }
            } else {                // B[kk = (r,s,k)][c] = w[k][r][s][c]
#pragma unroll
                for (int i = 0; i < PB; ++i) {
                    const int b = t + i * NT;
                    const int kq = (b / CGB) * 4;
                    int k = c0 + kq, r = r0, sx = s0;
                    while (k >= CC) { k -= CC; if (++sx == g.S) { sx = 0; ++r; } }
#pragma unroll
                    for (int jr = 0; jr < 4; ++jr) {
                        if (jr > 0 && ++k == CC) { k = 0; if (++sx == g.S) { sx = 0; ++r; } }
                        const bool ok = b < NBB && bcol_ok && k0 + kq + jr < kend_i;
                        const long off = (((long)k * g.R + r) * g.S + sx) * g.C + bcol_c;
                        rb_m[s][4 * i + jr] = ld8(Bm + (ok ? off : 0));
                        mb_m[s][4 * i + jr] = ok;
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < PA; ++i) {  // A[kk][m] = dy[kk][m]
                const int b = t + i * NT;
                const int kq = (b / CGA) * 4;
#pragma unroll
                for (int jr = 0; jr < 4; ++jr) {
                    const int kk = k0 + kq + jr;
                    const bool ok = b < NBA && kk < kend_i && acol < args.M;
                    ra_m[s][4 * i + jr] = ld8(Bm + (ok ? (long)kk * g.K + acol : 0));
                    ma_m[s][4 * i + jr] = ok;
                }
            }
            // B[kk = (n,p,q)][j = (r,s,c)] = x[n, p*st-pad+r, q*st-pad+s, c]
            const int q0 = k0 % g.Q;
            const int t0 = k0 / g.Q;
            const int p0 = t0 % g.P;
            const int n0i = t0 / g.P;
#pragma unroll
            for (int i = 0; i < PB; ++i) {
                const int b = t + i * NT;
                const int kq = (b / CGB) * 4;
                int q = q0 + kq, p = p0, n = n0i;
                while (q >= g.Q) { q -= g.Q; if (++p == g.P) { p = 0; ++n; } }
#pragma unroll
                for (int jr = 0; jr < 4; ++jr) {
                    if (jr > 0 && ++q == g.Q) { q = 0; if (++p == g.P) { p = 0; ++n; } }
                    const int h = p * g.st - g.pad + bcol_r;
                    const int w = q * g.st - g.pad + bcol_s;
                    const bool ok = b < NBB && bcol_ok && k0 + kq + jr < kend_i &&
                                    (unsigned)h < (unsigned)g.H && (unsigned)w < (unsigned)g.W;
                    const long off = (((long)n * g.H + h) * g.W + w) * g.C + bcol_c;
                    rb_m[s][4 * i + jr] = ld8(A + (ok ? off : 0));
                    mb_m[s][4 * i + jr] = ok;
                }
            }
        }
    };

    // column c (0..3) of four 4-element rows, as two (row j, row j+1) pairs
    auto col_pairs = [](const uintx2* rows, int c) -> uintx2 {
        auto el = [&](int j) -> unsigned {
            const unsigned w = (c < 2) ? rows[j].x : rows[j].y;
            return (c & 1) ? (w >> 16) : (w & 0xFFFFu);
        };
        return uintx2{el(0) | (el(1) << 16), el(2) | (el(3) << 16)};
    };

    auto sstore = [&](auto S) {
        constexpr int s = decltype(S)::value;
        unsigned short* As = smem + s * (BM + BN) * LDX;
        unsigned short* Bs = As + BM * LDX;
        const uintx4 z4{0u, 0u, 0u, 0u};
        const uintx2 z2{0u, 0u};
        if constexpr (A_KMAJ) {
#pragma unroll
            for (int i = 0; i < GA; ++i) {
                const int row = t / KG + i * (NT / KG);
                *reinterpret_cast<uintx4*>(As + row * LDX + kg) = ma_k[s][i] ? ra_k[s][i] : z4;
            }
        } else {
#pragma unroll
            for (int i = 0; i < PA; ++i) {
                const int b = t + i * NT;
                if (b >= NBA) continue;
                const int kq = (b / CGA) * 4;
                uintx2 rows[4];
#pragma unroll
                for (int jr = 0; jr < 4; ++jr)
                    rows[jr] = ma_m[s][4 * i + jr] ? ra_m[s][4 * i + jr] : z2;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int col = (t % CGA) * 4 + c;
                    *reinterpret_cast<uintx2*>(As + col * LDX + kq) = col_pairs(rows, c);
                }
            }
        }
        if constexpr (B_KMAJ) {
#pragma unroll
            for (int i = 0; i < GB; ++i) {
                const int row = t / KG + i * (NT / KG);
                *reinterpret_cast<uintx4*>(Bs + row * LDX + kg) = mb_k[s][i] ? rb_k[s][i] : z4;
            }
        } else {
#pragma unroll
            for (int i = 0; i < PB; ++i) {
                const int b = t + i * NT;
                if (b >= NBB) continue;
                const int kq = (b / CGB) * 4;
                uintx2 rows[4];
#pragma unroll
                for (int jr = 0; jr < 4; ++jr)
                    rows[jr] = mb_m[s][4 * i + jr] ? rb_m[s][4 * i + jr] : z2;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int col = (t % CGB) * 4 + c;
                    *reinterpret_cast<uintx2*>(Bs + col * LDX + kq) = col_pairs(rows, c);
                }
            }
        }
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int lr = lane & 31;
    const int lk = lane >> 5;
    // one k tile: prefetch tile kt+2 into register set s, multiply LDS buffer
    // s, write tile kt+1 (register set s^1) to LDS buffer s^1.  The loads are
    // unconditional (a tile past the end is all masked): with every load on
    // one path the compiler's wait before the LDS write counts only the
    // older set.
    auto step = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        gload(kt + 2, S);
        const unsigned short* As = smem + s * (BM + BN) * LDX;
        const unsigned short* Bs = As + BM * LDX;
        __builtin_amdgcn_s_setprio(1);
        if (kt < ktiles) {
#pragma unroll
        for (int kk = 0; kk < BKX; kk += 16) {
            bf16x8 av[TM], bv[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                av[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(
                                                       As + (wm + 32 * i + lr) * LDX + kk + 8 * lk));
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bv[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(
                                                       Bs + (wn + 32 * j + lr) * LDX + kk + 8 * lk));
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0,
                                                                         0, 0);
        }
        }
        __builtin_amdgcn_s_setprio(0);
        if (kt + 1 < ktiles) sstore(std::integral_constant<int, s ^ 1>{});
        __syncthreads();
    };

    const std::integral_constant<int, 0> I0{};
    const std::integral_constant<int, 1> I1{};
    gload(0, I0);
    gload(1, I1);
    if (ktiles > 0) sstore(I0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; kt += 2) {
        step(kt, I0);
        step(kt + 1, I1);
    }
    static_assert(sizeof(smem) >= (NT / 64) * SLOT_FLOATS * sizeof(float), "epilogue slots");
    write_tile<BM, BN, TM, TN>(args, wk, acc, wm, wn, lane,
                               reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS,
                               reinterpret_cast<float*>(smem));
}

// ---- bf16 kernel on k-major bf16 operands -------------------------------------
// Forward and stride-1 or stride-2 data-gradient contractions whose
// reduction channel count (C forward, K data gradient) is a multiple of the
// k tile, so that one k tile is one kernel tap (r, s) and BKX consecutive
// channels.  Both operands
// are k-major: A rows are gathered pixels (the implicit im2col of x; for the
// data gradient, of dy, where the tap enters with the opposite sign), B rows
// are weight rows (w [K][R][S][C] forward, its transposed copy [C][R][S][K]
// for the data gradient).  Operands are read with buffer loads, whose range
// check returns zeros for an offset past the end of the buffer: a lane whose
// pixel lies in the padding, or whose row lies past the matrix, gets such an
// offset, so staging needs no masks and a row's byte offset changes per tile
// only by the tap term.  A stride-2 data gradient reads dy pixel (h/2, w/2)
// of x pixel (h, w) shifted by the tap when both are even, and nothing
// otherwise.  Same LDS layout, MFMA loop and two-tile-deep staging as
// igemm_h16_kernel.

template <int OP, int BM, int BN, int WM, int WN, int BKX>
__global__ void __launch_bounds__(64 * (BM / WM) * (BN / WN), 2) igemm_h16k_kernel(KArgs args) {
    static_assert(OP == OP_FWD || OP == OP_DGRAD, "k-major operands");
    constexpr int NT = 64 * (BM / WM) * (BN / WN);
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int LDX = BKX + 8;
    constexpr int WAVES_N = BN / WN;
    constexpr int KG = BKX / 8;                  // 8-k groups per row
    constexpr int GA = BM * KG / NT;             // A groups per thread
    constexpr int GB = BN * KG / NT;
    static_assert(BKX % 16 == 0 && GA >= 1 && GB >= 1 && NT % KG == 0 &&
                  (BM * KG) % NT == 0 && (BN * KG) % NT == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) unsigned short smem[2 * (BM + BN) * LDX];

    const ConvGeo& g = args.g;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int wm = (wave / WAVES_N) * WM;
    const int wn = (wave % WAVES_N) * WN;
    const Work wk = decode_work<BM, BN>(args);
    const int ktiles = (int)((wk.kend - wk.kbeg) / BKX);   // whole tiles by construction
    const int kg = (t % KG) * 8;
    // image and channel count of the gathered operand
    const int IH = (OP == OP_FWD) ? g.H : g.P;
    const int IW = (OP == OP_FWD) ? g.W : g.Q;
    const int CC = (OP == OP_FWD) ? g.C : g.K;
    const unsigned a_bytes = (unsigned)((long)g.N * IH * IW * CC * 2);
    const unsigned b_bytes = (unsigned)(args.Ncols * args.Kred * 2);
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(args.a16), (short)0, (int)a_bytes, BUF_CFG);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(args.b16), (short)0, (int)b_bytes, BUF_CFG);

    // A row i: pixel of tap (0, 0) and its element offset (channel kg); for
    // a stride-2 data gradient the offset of the image's first pixel instead
    const bool st2 = (OP == OP_DGRAD) && g.st == 2;
    int a_h[GA], a_w[GA], a_off[GA];
    bool a_ok[GA];
#pragma unroll
    for (int i = 0; i < GA; ++i) {
        const long m = wk.m0 + t / KG + i * (NT / KG);
        a_ok[i] = m < args.M;
        const long mm = a_ok[i] ? m : 0;
        int n, h0, w0;
        if constexpr (OP == OP_FWD) {
            const int q = (int)(mm % g.Q); const long tt = mm / g.Q;
            const int p = (int)(tt % g.P); n = (int)(tt / g.P);
            h0 = p * g.st - g.pad;
            w0 = q * g.st - g.pad;
        } else {
            const int w = (int)(mm % g.W); const long tt = mm / g.W;
            const int h = (int)(tt % g.H); n = (int)(tt / g.H);
            h0 = h + g.pad;
            w0 = w + g.pad;
        }
        a_h[i] = h0;
        a_w[i] = w0;
        a_off[i] = st2 ? n * IH * IW * CC + kg : ((n * IH + h0) * IW + w0) * CC + kg;
    }
    // B row i: byte offset of its first k (the tile's k enters as soffset)
    unsigned b_off[GB];
#pragma unroll
    for (int i = 0; i < GB; ++i) {
        const long n = wk.n0 + t / KG + i * (NT / KG);
        b_off[i] = n < args.Ncols ? (unsigned)((n * args.Kred + kg) * 2) : BUF_OOB;
    }

    uintx4 ra[2][GA], rb[2][GB];
    // tap (tr, ts) and channel base tc of the next tile to load.  The tiles
    // go channel chunk by channel chunk, all R*S taps of a chunk in a row
    // (tile T = chunk T / RS, tap T % RS): the tap-shifted reads of the same
    // BKX channels follow each other and hit in the caches.
    const int RSN = g.R * g.S;
    int tc, tr, ts;
    {
        const int T0 = (int)(wk.kbeg / BKX);
        tc = (T0 / RSN) * BKX;
        const int rs = T0 % RSN;
        tr = rs / g.S;
        ts = rs - tr * g.S;
    }

    // Loads of tiles past the end are harmless: every offset is range-checked
    // and such a tile is never written to LDS.
    auto gload = [&](auto S) {
        constexpr int s = decltype(S)::value;
        const int dr = (OP == OP_FWD) ? tr : -tr;
        const int ds = (OP == OP_FWD) ? ts : -ts;
        const int sk = (dr * IW + ds) * CC + tc;
#pragma unroll
        for (int i = 0; i < GA; ++i) {
            const int h = a_h[i] + dr, w = a_w[i] + ds;
            if (st2) {
                // dy pixel (h / 2, w / 2) when both are even (a tap on the stride grid)
                const bool ok = a_ok[i] && ((h | w) & 1) == 0 && h >= 0 && w >= 0 &&
                                (h >> 1) < IH && (w >> 1) < IW;
                const int off = a_off[i] + ((h >> 1) * IW + (w >> 1)) * CC + tc;
                ra[s][i] = buf_load16(rsA, ok ? (unsigned)off * 2u : BUF_OOB, 0u);
            } else {
                const bool ok = a_ok[i] && (unsigned)h < (unsigned)IH && (unsigned)w < (unsigned)IW;
                ra[s][i] = buf_load16(rsA, ok ? (unsigned)(a_off[i] + sk) * 2u : BUF_OOB, 0u);
            }
        }
        const unsigned kload = (unsigned)((tr * g.S + ts) * CC + tc);   // linear reduction index
#pragma unroll
        for (int i = 0; i < GB; ++i) rb[s][i] = buf_load16(rsB, b_off[i], kload * 2u);
        if (++ts == g.S) {
            ts = 0;
            if (++tr == g.R) { tr = 0; tc += BKX; }
        }
    };

    auto sstore = [&](auto S) {
        constexpr int s = decltype(S)::value;
        unsigned short* As = smem + s * (BM + BN) * LDX;
        unsigned short* Bs = As + BM * LDX;
#pragma unroll
        for (int i = 0; i < GA; ++i)
            *reinterpret_cast<uintx4*>(As + (t / KG + i * (NT / KG)) * LDX + kg) = ra[s][i];
#pragma unroll
        for (int i = 0; i < GB; ++i)
            *reinterpret_cast<uintx4*>(Bs + (t / KG + i * (NT / KG)) * LDX + kg) = rb[s][i];
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int lr = lane & 31;
    const int lk = lane >> 5;
    auto step = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        gload(S);                                  // tile kt + 2
        const unsigned short* As = smem + s * (BM + BN) * LDX;
        const unsigned short* Bs = As + BM * LDX;
        __builtin_amdgcn_s_setprio(1);
        if (kt < ktiles) {
#pragma unroll
            for (int kk = 0; kk < BKX; kk += 16) {
                bf16x8 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    av[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(
                                                           As + (wm + 32 * i + lr) * LDX + kk + 8 * lk));
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    bv[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(
                                                           Bs + (wn + 32 * j + lr) * LDX + kk + 8 * lk));
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j],
                                                                             acc[i][j], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        if (kt + 1 < ktiles) sstore(std::integral_constant<int, s ^ 1>{});
        __syncthreads();
    };

    const std::integral_constant<int, 0> I0{};
    const std::integral_constant<int, 1> I1{};
    gload(I0);
    gload(I1);
    if (ktiles > 0) sstore(I0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; kt += 2) {
        step(kt, I0);
        step(kt + 1, I1);
    }
    static_assert(sizeof(smem) >= (NT / 64) * SLOT_FLOATS * sizeof(float), "epilogue slots");
    write_tile<BM, BN, TM, TN>(args, wk, acc, wm, wn, lane,
                               reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS,
                               reinterpret_cast<float*>(smem));
}


// ---- bf16 k-major contraction with operands loaded straight into LDS ---------
// The forward and stride-1 data-gradient contractions of igemm_h16k_kernel on
// a 256 x 128 workgroup tile of four waves, one per SIMD, each owning a
// 128 x 64 block as 4 x 2 MFMA 32x32x16 tiles: per 16-deep k step a wave reads
// 6 operand fragments from LDS for 8 MFMAs, where the 32 x 64 waves of
// igemm_h16k_kernel read 3 for 2.  Operands go from memory into LDS directly
// (buffer_load_dwordx4 ... lds: lane l of a wave writes 16 bytes at the wave's
// LDS base + 16 l), range-checked like the other buffer loads (padding taps
// and rows past the matrix read zeros), so no registers stage them.
//
// A k tile is 32 reduction indices (64 bytes per row, four 16-byte chunks),
// taken channel chunk by channel chunk with all taps of a chunk in a row, as in
// igemm_h16k_kernel; the tap and chunk of the next tile to load are stepped,
// not divided out.  One load instruction fills 16 rows; the lane that lands in
// chunk position p of row r loads chunk p ^ ((r / 4) mod 4) of that row, so
// the operand reads of consecutive rows at one chunk fall in distinct bank
// groups.  Four LDS stages, each its own array (so the compiler's wait
// counters tell them apart), A rows then B rows.
//
// With one wave per SIMD a wave issues at most one instruction per four
// clocks, eight per MFMA 32x32x16, and nothing else hides its latencies, so
// the k loop is lean and software-pipelined by hand.  Which taps of each A
// row lie inside the image is a bit mask computed once, so a load costs three
// vector operations; the steady-state steps carry no conditions.  Each tile is
// two 16-deep halves; the operands of one half are read from LDS while the
// products of the other run (the reads spread between the MFMAs).  In the
// middle of tile kt, between its halves, the wave waits for its own loads of
// tile kt+1, a barrier makes every wave's loads of kt+1 visible and tells that
// all reads of tile kt-1 are done, the loads of tile kt+3 go into kt-1's
// stage, and the first half of kt+1 is read during the second half's products
// of kt.  A load thus has two tiles' time to land.
constexpr int H16D_BM = 256, H16D_BN = 128, H16D_BK = 32, H16D_WAVES = 4, H16D_STAGES = 3;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    // s_waitcnt vmcnt(N), expcnt and lgkmcnt not waited for (gfx9 encoding)
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// 16 bytes per lane from a buffer straight into LDS: lane l writes at lds + 16 l
// (the LDS byte address goes in M0, which must be uniform).  Written as
// assembly so that the compiler does not track these loads: the kernel waits
// for them itself (wait_vmcnt before the barrier that publishes a stage), and
// the compiler's own tracking, which cannot tell the stages apart across the
// loop's back edge, would wait for every load in flight before the next
// stage's LDS reads.  The memory clobber keeps LDS accesses on their side.
__device__ __forceinline__ void buf_load16_lds(__amdgpu_buffer_rsrc_t rs, void* lds, unsigned voff,
                                               unsigned soff) {
    const unsigned m0 = (unsigned)(size_t)(lds_ptr_t)lds;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(m0), "v"(voff), "s"(rs), "s"(soff)
                 : "memory", "m0");
}

// s_barrier without a memory fence (no wait for outstanding loads); the asm
// memory clobber keeps the compiler from moving LDS accesses across it
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// scheduling hint for one block of straight-line code: R LDS reads spread
// evenly among M MFMAs, each read after its share of MFMAs
template <int M, int R, int Q = 0>
__device__ __forceinline__ void interleave_mfma_reads() {
    if constexpr (Q < R) {
        constexpr int n = (Q + 1) * M / R - Q * M / R;
        if constexpr (n > 0) __builtin_amdgcn_sched_group_barrier(0x008, n, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        interleave_mfma_reads<M, R, Q + 1>();
    }
}

template <int OP>
__global__ void __launch_bounds__(64 * H16D_WAVES, 2) igemm_h16d_kernel(KArgs args) {
    static_assert(OP == OP_FWD || OP == OP_DGRAD, "k-major operands");
    constexpr int BM = H16D_BM, BN = H16D_BN, BK = H16D_BK, ROW = 2 * BK, NW = H16D_WAVES;
    constexpr int WM = BM / 2, WN = BN / 2, TM = WM / 32, TN = WN / 32;
    constexpr int LA = BM / 16 / NW, LB = BN / 16 / NW;   // load instructions per wave per tile
    constexpr int LPT = LA + LB;
    constexpr int SB = (BM + BN) * ROW;                    // one stage: A rows, then B rows
    constexpr int NS = H16D_STAGES;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[NS * SB];

    const ConvGeo& g = args.g;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = (wave >> 1) * WM;
    const int wn = (wave & 1) * WN;
    const Work wk = decode_work<BM, BN>(args);
    const int ktiles = (int)((wk.kend - wk.kbeg) / BK);   // whole tiles by construction
    const int T0 = (int)(wk.kbeg / BK);
    const int IH = (OP == OP_FWD) ? g.H : g.P;
    const int IW = (OP == OP_FWD) ? g.W : g.Q;
    const int CC = (OP == OP_FWD) ? g.C : g.K;
    const int RSN = g.R * g.S;                             // at most 32 (the tap masks)
    const unsigned a_bytes = (unsigned)((long)g.N * IH * IW * CC * 2);
    const unsigned b_bytes = (unsigned)(args.Ncols * args.Kred * 2);
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(args.a16), (short)0, (int)a_bytes, BUF_CFG);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(args.b16), (short)0, (int)b_bytes, BUF_CFG);

    // the chunk this lane loads: position lane % 4 of row (.. + lane / 4),
    // swizzled by (row / 4) mod 4 = (lane / 16) mod 4
    const int kc = ((lane & 3) ^ ((lane >> 4) & 3)) * 8;
    // A rows: byte offset of the row's pixel at tap (0, 0) and chunk kc,
    // and the taps (bit r*S + s) whose pixel lies outside the image (all of
    // them for rows past M)
    int a_off[LA];
    unsigned a_out[LA];
#pragma unroll
    for (int j = 0; j < LA; ++j) {
        const long m = wk.m0 + (wave * LA + j) * 16 + (lane >> 2);
        const bool row_ok = m < args.M;
        const long mm = row_ok ? m : 0;
        int n, h0, w0;
        if constexpr (OP == OP_FWD) {
            const int q = (int)(mm % g.Q); const long tt = mm / g.Q;
            const int p = (int)(tt % g.P); n = (int)(tt / g.P);
            h0 = p * g.st - g.pad;
            w0 = q * g.st - g.pad;
        } else {
            const int w = (int)(mm % g.W); const long tt = mm / g.W;
            const int h = (int)(tt % g.H); n = (int)(tt / g.H);
            h0 = h + g.pad;
            w0 = w + g.pad;
        }
        unsigned out = 0;
        for (int r = 0; r < g.R; ++r)
            for (int s = 0; s < g.S; ++s) {
                const int h = (OP == OP_FWD) ? h0 + r : h0 - r;
                const int w = (OP == OP_FWD) ? w0 + s : w0 - s;
                if (!row_ok || (unsigned)h >= (unsigned)IH || (unsigned)w >= (unsigned)IW)
                    out |= 1u << (r * g.S + s);
            }
        a_out[j] = out;
        a_off[j] = (((n * IH + h0) * IW + w0) * CC + kc) * 2;
    }
    unsigned b_off[LB];
#pragma unroll
    for (int j = 0; j < LB; ++j) {
        const long n = wk.n0 + (wave * LB + j) * 16 + (lane >> 2);
        b_off[j] = n < args.Ncols ? (unsigned)((n * args.Kred + kc) * 2) : BUF_OOB;
    }

    // the next tile to load, in reduction order (chunk T / RS, tap T % RS):
    // tap (ir, is), index itap = ir * S + is, of channel chunk ic
    const int rs0 = T0 % RSN;
    int ic = (T0 / RSN) * BK, ir = rs0 / g.S, is = rs0 - ir * g.S, itap = rs0;
    auto issue = [&](unsigned char* S) __attribute__((always_inline)) {
        const int dr = (OP == OP_FWD) ? ir : -ir;
        const int ds = (OP == OP_FWD) ? is : -is;
        const int sk2 = ((dr * IW + ds) * CC + ic) * 2;
#pragma unroll
        for (int j = 0; j < LA; ++j) {
            // a tap outside the image sets bit 31: past the end of any operand
            // (only bit 0 of the shifted mask survives the shift by 31)
            buf_load16_lds(rsA, S + (wave * LA + j) * 1024,
                           ((a_out[j] >> itap) << 31) | (unsigned)(a_off[j] + sk2), 0u);
        }
        const int kload = (itap * CC + ic) * 2;
#pragma unroll
        for (int j = 0; j < LB; ++j)
            buf_load16_lds(rsB, S + BM * ROW + (wave * LB + j) * 1024, b_off[j], (unsigned)kload);
        ++itap;
        if (++is == g.S) {
            is = 0;
            if (++ir == g.R) { ir = 0; itap = 0; ic += BK; }
        }
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int lr = lane & 31, lk = lane >> 5;
    const int rsw = (lr >> 2) & 3;       // swizzle of this lane's operand rows
    // operand offsets of half 0 and half 1 of a tile within a stage
    const int oa0 = (wm + lr) * ROW + ((0 + lk) ^ rsw) * 16;
    const int oa1 = (wm + lr) * ROW + ((2 + lk) ^ rsw) * 16;
    const int ob0 = BM * ROW + (wn + lr) * ROW + ((0 + lk) ^ rsw) * 16;
    const int ob1 = BM * ROW + (wn + lr) * ROW + ((2 + lk) ^ rsw) * 16;
    bf16x8 a0[TM], b0[TN], a1[TM], b1[TN];
    auto lds16 = [](const unsigned char* p) __attribute__((always_inline)) {
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uintx4*>(p));
    };
    auto read_half = [&](const unsigned char* S, int oa, int ob, bf16x8 (&a)[TM], bf16x8 (&b)[TN])
        __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = lds16(S + oa + 32 * i * ROW);
#pragma unroll
        for (int j = 0; j < TN; ++j) b[j] = lds16(S + ob + 32 * j * ROW);
    };
    auto mma_half = [&](const bf16x8 (&a)[TM], const bf16x8 (&b)[TN]) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };

    // tile kt sits in stage `cur`, kt+1 in `nxt`; `fill` (kt-1's stage)
    // receives tile kt+NS-1.  On entry a0/b0 hold the first half of tile kt.
    // A steady step: tiles kt+1 .. kt+NS-1 all exist.
    auto step_full = [&](const unsigned char* cur, const unsigned char* nxt, unsigned char* fill)
        __attribute__((always_inline)) {
        read_half(cur, oa1, ob1, a1, b1);
        mma_half(a0, b0);
        interleave_mfma_reads<TM * TN, TM + TN>();
        wait_vmcnt<(NS - 3) * LPT>();
        lds_barrier();
        issue(fill);
        read_half(nxt, oa0, ob0, a0, b0);
        mma_half(a1, b1);
        interleave_mfma_reads<TM * TN, TM + TN>();
    };
    // one of the last steps: tiles past the end are neither waited for nor
    // loaded (outstanding after the wait: the existing tiles kt+2 .. kt+NS-2)
    auto step_tail = [&](int kt, const unsigned char* cur, const unsigned char* nxt,
                         unsigned char* fill) __attribute__((always_inline)) {
        read_half(cur, oa1, ob1, a1, b1);
        mma_half(a0, b0);
        if (kt + 1 < ktiles) {
            if (NS == 4 && kt + 2 < ktiles) wait_vmcnt<LPT>();
            else wait_vmcnt<0>();
            lds_barrier();
            if (kt + NS - 1 < ktiles) issue(fill);
            read_half(nxt, oa0, ob0, a0, b0);
        }
        mma_half(a1, b1);
    };
    static_assert(NS == 3 || NS == 4, "stages");
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < ktiles) issue(smem + s * SB);
    if (ktiles > 0) {
        if (NS == 4 && ktiles > 2) wait_vmcnt<2 * LPT>();
        else if (ktiles > 1) wait_vmcnt<LPT>();
        else wait_vmcnt<0>();
        lds_barrier();
        read_half(smem, oa0, ob0, a0, b0);
    }
    int kt = 0;
    for (; kt + NS - 1 + (NS - 1) < ktiles; kt += NS) {
#pragma unroll
        for (int s = 0; s < NS; ++s)
            step_full(smem + s * SB, smem + ((s + 1) % NS) * SB, smem + ((s + NS - 1) % NS) * SB);
    }
    for (; kt < ktiles; ++kt) {
        const int s = kt % NS;
        step_tail(kt, smem + s * SB, smem + ((s + 1) % NS) * SB, smem + ((s + NS - 1) % NS) * SB);
    }
    __syncthreads();
    // the epilogue's per-wave 4 KB slots, in the first stage
    static_assert(SB >= NW * SLOT_FLOATS * (int)sizeof(float), "epilogue slots");
    float* slot = reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS;
    write_tile_plain<BM, BN, TM, TN, true>(args, wk, acc, wm, wn, lane, slot);
}


// ---- bf16 weight-gradient kernel on m-major LDS tiles --------------------------
// out[k][(r,s,c)] = sum over output pixels (n,p,q) of dy[(n,p,q)][k] *
// x[n, p*st-pad+r, q*st-pad+s, c].  Both operands have the reduction index
// (the pixel) as their memory row, so both are staged m-major: a k tile is
// BKX pixel rows of BM output channels of dy and BN im2col columns of x, each
// row segment copied with 16-byte buffer loads as it lies in memory (8
// consecutive channels; C % 8 == 0 keeps them within one tap).  The MFMA
// operand of a lane (8 consecutive k of one row) is read with two LDS
// transpose reads (ds_read_b64_tr_b16): in every group of 16 lanes, lane i
// receives element i mod 4 of the 8 bytes read by lane 4e + i/4 as its value
// e, so when source lane S reads k row k0 + S/4 at columns m0 + 4 (S mod 4),
// lane i holds k0..k0+3 of column m0 + i.  The LDS serves an 8-byte read
// 32 lanes at a time from 64 four-byte banks; those 32 lanes read 16
// consecutive dwords of each of four rows, so rows are padded by 32 elements
// (a pitch of 16 mod 64 dwords for BM = 128, 48 for BM = 64), which puts the
// four rows in disjoint quarters of the banks.  The
// output pixel of a k row is divided into (n, p, q) by multiply-high with
// constants computed on the host.
template <int BM, int BN, int WM, int WN, int BKX>
__global__ void __launch_bounds__(64 * (BM / WM) * (BN / WN), 2) igemm_h16w_kernel(KArgs args) {
    constexpr int NT = 64 * (BM / WM) * (BN / WN);
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int PA = BM + 32, PB = BN + 32;    // LDS row pitch (bf16)
    constexpr int WAVES_N = BN / WN;
    constexpr int CGA = BM / 8, CGB = BN / 8;    // 16-byte groups per row
    constexpr int LA = BKX * CGA / NT;           // loads per thread per tile
    constexpr int LB = BKX * CGB / NT;
    static_assert(BKX % 16 == 0 && LA >= 1 && LB >= 1 && (BKX * CGA) % NT == 0 &&
                  (BKX * CGB) % NT == 0 && NT % CGA == 0 && NT % CGB == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) unsigned short smem[2 * BKX * (PA + PB)];

    const ConvGeo& g = args.g;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int wm = (wave / WAVES_N) * WM;
    const int wn = (wave % WAVES_N) * WN;
    const Work wk = decode_work<BM, BN>(args);
    const int ktiles = (int)((wk.kend - wk.kbeg + BKX - 1) / BKX);
    const int kend = (int)wk.kend;
    const unsigned x_bytes = (unsigned)((long)g.N * g.H * g.W * g.C * 2);
    const unsigned dy_bytes = (unsigned)((long)g.N * g.P * g.Q * g.K * 2);
    const __amdgpu_buffer_rsrc_t rsX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(args.a16), (short)0, (int)x_bytes, BUF_CFG);
    const __amdgpu_buffer_rsrc_t rsD = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(args.b16), (short)0, (int)dy_bytes, BUF_CFG);

    // dy: this thread's column group and row of each load
    const int acol = (t % CGA) * 8;
    const bool acol_ok = wk.m0 + acol < args.M;
    const unsigned a_voff = (unsigned)(wk.m0 + acol) * 2u;
    int arow[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) arow[i] = (t + i * NT) / CGA;
    // x: this thread's column group = one tap (r, s) and 8 channels from c
    const int bcol = (t % CGB) * 8;
    const long jb = wk.n0 + bcol;
    const bool bcol_ok = jb < args.Ncols;
    int bc, br, bs;
    {
        const long jj = bcol_ok ? jb : 0;
        bc = (int)(jj % g.C);
        const int rs = (int)(jj / g.C);
        br = rs / g.S;
        bs = rs - br * g.S;
    }
    int brow[LB];
#pragma unroll
    for (int i = 0; i < LB; ++i) brow[i] = (t + i * NT) / CGB;

    uintx4 ra[2][LA], rb[2][LB];

    // loads of tile kt (rows past kend, including whole tiles past the end,
    // read zeros through the range check)
    auto gload = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        const int k0 = (int)wk.kbeg + kt * BKX;
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const int pix = k0 + arow[i];
            const bool ok = acol_ok && pix < kend;
            ra[s][i] = buf_load16(rsD, ok ? (unsigned)pix * (unsigned)(g.K * 2) + a_voff : BUF_OOB, 0u);
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const unsigned pix = (unsigned)(k0 + brow[i]);
            const unsigned t2 = (unsigned)(((unsigned long long)pix * args.mq) >> args.sq);
            const int q = (int)(pix - t2 * (unsigned)g.Q);
            const unsigned n = (unsigned)(((unsigned long long)t2 * args.mp) >> args.sp);
            const int p = (int)(t2 - n * (unsigned)g.P);
            const int h = p * g.st - g.pad + br;
            const int w = q * g.st - g.pad + bs;
            const bool ok = bcol_ok && (int)pix < kend && (unsigned)h < (unsigned)g.H &&
                            (unsigned)w < (unsigned)g.W;
            const int off = (((int)n * g.H + h) * g.W + w) * g.C + bc;
            rb[s][i] = buf_load16(rsX, ok ? (unsigned)off * 2u : BUF_OOB, 0u);
        }
    };

    auto sstore = [&](auto S) {
        constexpr int s = decltype(S)::value;
        unsigned short* As = smem + s * BKX * (PA + PB);
        unsigned short* Bs = As + BKX * PA;
#pragma unroll
        for (int i = 0; i < LA; ++i)
            *reinterpret_cast<uintx4*>(As + arow[i] * PA + acol) = ra[s][i];
#pragma unroll
        for (int i = 0; i < LB; ++i)
            *reinterpret_cast<uintx4*>(Bs + brow[i] * PB + bcol) = rb[s][i];
    };

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // transpose-read addressing: source lane S = lane % 16 of group gq = lane / 16
    // reads k row 8 (gq / 2) + S / 4 (+4 for the second half) at column
    // 16 (gq % 2) + 4 (S % 4) of a 32-column fragment
    const int gq = lane >> 4, sl = lane & 15;
    const int tr_row = 8 * (gq >> 1) + (sl >> 2);
    const int tr_col = 16 * (gq & 1) + 4 * (sl & 3);
    typedef short v4s __attribute__((ext_vector_type(4)));
    auto tr_read = [](const unsigned short* p) -> v4s {
        return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4s*)(
                (__attribute__((address_space(3))) unsigned short*)(p)));
    };
    auto frag = [&](const unsigned short* base, int pitch, int kk, int col) -> bf16x8 {
        const unsigned short* p = base + (kk + tr_row) * pitch + col + tr_col;
        const v4s lo = tr_read(p);
        const v4s hi = tr_read(p + 4 * pitch);
        typedef short v8s __attribute__((ext_vector_type(8)));
        const v8s v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(bf16x8, v);
    };

    auto step = [&](int kt, auto S) {
        constexpr int s = decltype(S)::value;
        gload(kt + 2, S);
        const unsigned short* As = smem + s * BKX * (PA + PB);
        const unsigned short* Bs = As + BKX * PA;
        __builtin_amdgcn_s_setprio(1);
        if (kt < ktiles) {
#pragma unroll
            for (int kk = 0; kk < BKX; kk += 16) {
                bf16x8 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) av[i] = frag(As, PA, kk, wm + 32 * i);
#pragma unroll
                for (int j = 0; j < TN; ++j) bv[j] = frag(Bs, PB, kk, wn + 32 * j);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j],
                                                                             acc[i][j], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        if (kt + 1 < ktiles) sstore(std::integral_constant<int, s ^ 1>{});
        __syncthreads();
    };

    const std::integral_constant<int, 0> I0{};
    const std::integral_constant<int, 1> I1{};
    gload(0, I0);
    gload(1, I1);
    if (ktiles > 0) sstore(I0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; kt += 2) {
        step(kt, I0);
        step(kt + 1, I1);
    }
    static_assert(sizeof(smem) >= (NT / 64) * SLOT_FLOATS * sizeof(float), "epilogue slots");
    write_tile<BM, BN, TM, TN>(args, wk, acc, wm, wn, lane,
                               reinterpret_cast<float*>(smem) + wave * SLOT_FLOATS,
                               reinterpret_cast<float*>(smem));
}



// Reduction of the cut tiles: workgroup = 64 elements of one tile x 16 split
// lanes; lane l adds splits l, l+16, ... (eight loads in flight at a time,
// added in split order), the lane sums are combined in a fixed order
// (deterministic), then the epilogue runs.
constexpr int SK_EL = 64, SK_LANES = 16, SK_BATCH = 8;

__global__ void __launch_bounds__(SK_EL * SK_LANES)
igemm_splitk_reduce_kernel(KArgs args, int BM, int BN) {
    __shared__ float red[SK_LANES][SK_EL];
    const int el = threadIdx.x % SK_EL;
    const int ln = threadIdx.x / SK_EL;
    const int chunks = (BM * BN) / SK_EL;
    const int rt = blockIdx.x / chunks;                 // index among the cut tiles
    const int e = (blockIdx.x - rt * chunks) * SK_EL + el;
    const int tile = args.tfull + rt;
    const long row = (long)(tile / args.tiles_n) * BM + e / BN;
    const long col = (long)(tile % args.tiles_n) * BN + e % BN;
    float s = 0.f;
    const float* src = args.ws + (long)rt * args.splits * (BM * BN) + e;
    for (int z0 = ln; z0 < args.splits; z0 += SK_LANES * SK_BATCH) {
        float v[SK_BATCH];
#pragma unroll
        for (int b = 0; b < SK_BATCH; ++b) {
            const int z = z0 + b * SK_LANES;
            v[b] = z < args.splits ? src[(long)z * (BM * BN)] : 0.f;
        }
#pragma unroll
        for (int b = 0; b < SK_BATCH; ++b) s += v[b];
    }
    red[ln][el] = s;
    __syncthreads();
    if (ln == 0 && row < args.M && col < args.Ncols) {
        float acc = 0.f;
        for (int l = 0; l < SK_LANES; ++l) acc += red[l][el];
        float* dst = out_ptr(args.out, args.bias_out, row, col, args.Ncols, args.epi);
        const float v = epilogue(acc, row, col, args.Ncols, args.epi, args.bias, args.mask, dst);
        *dst = v;
        if (args.out16) args.out16[row * args.Ncols + col] = bf16_bits(v);
    }
}

// The same reduction for at most 16 splits: one thread per 4 consecutive
// elements of the cut tiles; all of its split partials (one float4 each) are
// loaded before they are added, in split order.
__global__ void __launch_bounds__(256) igemm_cut_reduce_kernel(KArgs args, int BM, int BN) {
    const int tile_elems = BM * BN;
    const int per_tile = tile_elems / 4;
    const long total = (long)(args.tiles_m * args.tiles_n - args.tfull) * per_tile;
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (long)gridDim.x * blockDim.x) {
        const int rt = (int)(i / per_tile);
        const int e = (int)(i - (long)rt * per_tile) * 4;
        const int tile = args.tfull + rt;
        const long row = (long)(tile / args.tiles_n) * BM + e / BN;
        const long col0 = (long)(tile % args.tiles_n) * BN + e % BN;
        if (row >= args.M || col0 >= args.Ncols) continue;
        const float4* src =
            reinterpret_cast<const float4*>(args.ws + (long)rt * args.splits * tile_elems + e);
        float4 part[SK_LANES];
#pragma unroll
        for (int z = 0; z < SK_LANES; ++z)
            part[z] = z < args.splits ? src[(long)z * per_tile] : make_float4(0.f, 0.f, 0.f, 0.f);
        float4 acc = part[0];
#pragma unroll
        for (int z = 1; z < SK_LANES; ++z) {
            if (z < args.splits) {
                acc.x += part[z].x; acc.y += part[z].y; acc.z += part[z].z; acc.w += part[z].w;
            }
        }
        const float a4[4] = {acc.x, acc.y, acc.z, acc.w};
        float prev[4] = {0.f, 0.f, 0.f, 0.f};
        // epilogue reads first (see store_tile)
        if (args.epi & EPI_ACCUM) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (col0 + j < args.Ncols)
                    prev[j] = *out_ptr(args.out, args.bias_out, row, col0 + j, args.Ncols, args.epi);
        }
        const int epi = args.epi;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const long col = col0 + j;
            if (col >= args.Ncols) break;
            float v = a4[j];
            if (epi & EPI_BIAS) v += args.bias[col];
            if (epi & EPI_RELU) v = fmaxf(v, 0.f);
            if ((epi & EPI_MASK) && !(args.mask[row * args.Ncols + col] > 0.f)) v = 0.f;
            if (epi & EPI_ACCUM) v += prev[j];
            *out_ptr(args.out, args.bias_out, row, col, args.Ncols, epi) = v;
            if (args.out16) args.out16[row * args.Ncols + col] = bf16_bits(v);
        }
    }
}

// Reduction of the cut tiles with column statistics (a following batch norm):
// one workgroup per cut tile; thread = 4 consecutive columns x every RG-th
// row.  Each output is the sum of its split partials in split order plus the
// bias; the tile's column means and sums of squared deviations are then
// formed from the values kept in registers, exactly as tile_stats does for
// whole tiles.
constexpr int CRS_THREADS = 256, CRS_ROWS = 16;   // rows per thread at most

__global__ void __launch_bounds__(CRS_THREADS) igemm_cut_reduce_stats_kernel(KArgs args, int BM,
                                                                             int BN) {
    __shared__ float part[CRS_THREADS * 4];
    __shared__ float mean[256];
    const int CG = BN / 4, RG = CRS_THREADS / CG;
    const int t = threadIdx.x;
    const int cg = t % CG, rg = t / CG;
    const int rt = blockIdx.x;
    const int tile = args.tfull + rt;
    const long m0 = (long)(tile / args.tiles_n) * BM, n0 = (long)(tile % args.tiles_n) * BN;
    const long rows = min((long)BM, args.M - m0);
    const long col0 = n0 + 4 * cg;
    const float* src = args.ws + (long)rt * args.splits * BM * BN;
    float b4[4] = {0.f, 0.f, 0.f, 0.f};
    if (args.epi & EPI_BIAS)
        for (int e = 0; e < 4; ++e)
            if (col0 + e < args.Ncols) b4[e] = args.bias[col0 + e];
    // the partials of one split for every row of this thread are loaded
    // together (CRS_ROWS loads in flight), then added; each element still
    // sums its splits in split order
    float4 acc[CRS_ROWS];
    auto load_split = [&](int z, float4 (&p)[CRS_ROWS]) {
        const float* sz = src + (long)z * BM * BN + 4 * cg;
#pragma unroll
        for (int q = 0; q < CRS_ROWS; ++q) {
            const int r = rg + q * RG;
            p[q] = (r < BM && r < rows) ? *reinterpret_cast<const float4*>(sz + r * BN)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    load_split(0, acc);
    for (int z = 1; z < args.splits; ++z) {
        float4 p[CRS_ROWS];
        load_split(z, p);
#pragma unroll
        for (int q = 0; q < CRS_ROWS; ++q) {
            acc[q].x += p[q].x; acc[q].y += p[q].y; acc[q].z += p[q].z; acc[q].w += p[q].w;
        }
    }
    // 16-byte stores when the row length keeps them aligned
    const bool vec_out = (args.Ncols & 3) == 0 && col0 + 3 < args.Ncols &&
                         (((uintptr_t)args.out) & 15) == 0;
    float val[CRS_ROWS][4];
    float sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < CRS_ROWS; ++q) {
        const int r = rg + q * RG;
        for (int e = 0; e < 4; ++e) val[q][e] = 0.f;
        if (r >= BM || r >= rows) continue;
        val[q][0] = acc[q].x + b4[0];
        val[q][1] = acc[q].y + b4[1];
        val[q][2] = acc[q].z + b4[2];
        val[q][3] = acc[q].w + b4[3];
        float* o = args.out + (m0 + r) * args.Ncols + col0;
        if (vec_out) {
            *reinterpret_cast<float4*>(o) = make_float4(val[q][0], val[q][1], val[q][2], val[q][3]);
        } else {
            for (int e = 0; e < 4; ++e)
                if (col0 + e < args.Ncols) o[e] = val[q][e];
        }
        for (int e = 0; e < 4; ++e) sum[e] += val[q][e];
    }
    const long tm = m0 / BM;
    for (int pass = 0; pass < 2; ++pass) {
        if (pass == 1) {
            float mu[4];
            for (int e = 0; e < 4; ++e) { mu[e] = mean[4 * cg + e]; sum[e] = 0.f; }
#pragma unroll
            for (int q = 0; q < CRS_ROWS; ++q) {
                const int r = rg + q * RG;
                if (r >= BM || r >= rows) continue;
                for (int e = 0; e < 4; ++e) {
                    const float d = val[q][e] - mu[e];
                    sum[e] += d * d;
                }
            }
        }
        for (int e = 0; e < 4; ++e) part[(rg * CG + cg) * 4 + e] = sum[e];
        __syncthreads();
        if (rg == 0) {
            for (int e = 0; e < 4; ++e) {
                float s = 0.f;
                for (int g = 0; g < RG; ++g) s += part[(g * CG + cg) * 4 + e];
                const long col = col0 + e;
                if (pass == 0) {
                    mean[4 * cg + e] = rows > 0 ? s / (float)rows : 0.f;
                } else if (col < args.Ncols) {
                    args.stats[tm * args.Ncols + col] = mean[4 * cg + e];
                    args.stats[((long)args.tiles_m + tm) * args.Ncols + col] = s;
                }
            }
        }
        __syncthreads();
    }
}

struct KernelRef {
    const void* fn;
    int nt;
};

// Kernel families: fp32 operands staged from fp32 (vector width 1 or 4),
// bf16 rounded while staging from fp32 (1 or 4), bf16 operands in memory
// (general gather), bf16 operands in memory, both k-major (FWD and stride-1
// DGRAD with a reduction channel count that is a multiple of the k tile), and
// fp32 (vector width 4 or 1) with the wide epilogue.
// KF_F32_4F / KF_F32_4WF: the fp32 vector kernels in their FAST form (forward and
// stride-1 data gradient with a channel count that is a multiple of the k tile;
// weight gradient with an output width that is one).
enum { KF_F32_1, KF_F32_4, KF_BF_1, KF_BF_4, KF_H16, KF_H16K, KF_F32_4W, KF_F32_1W, KF_H16D,
       KF_F32_4F, KF_F32_4WF };

template <int OP, int CFG, int KF>
KernelRef kref() {
    constexpr TileCfg c = kCfgs[CFG];
    constexpr int nt = 64 * (c.bm / c.wm) * (c.bn / c.wn);
    if constexpr (KF == KF_H16K && OP != OP_WGRAD)
        return {reinterpret_cast<const void*>(
                    &igemm_h16k_kernel<OP, c.bm, c.bn, c.wm, c.wn, c.bkh>), nt};
    else if constexpr (KF == KF_H16K)
        return {reinterpret_cast<const void*>(
                    &igemm_h16w_kernel<c.bm, c.bn, c.wm, c.wn, c.bkh>), nt};
    else if constexpr (KF == KF_H16 || KF == KF_H16K)
        return {reinterpret_cast<const void*>(
                    &igemm_h16_kernel<OP, c.bm, c.bn, c.wm, c.wn, c.bkh>), nt};
    else if constexpr (KF == KF_BF_1 || KF == KF_BF_4)
        return {reinterpret_cast<const void*>(
                    &igemm_bf16_kernel<OP, c.bm, c.bn, c.wm, c.wn, KF == KF_BF_4 ? 4 : 1>), nt};
    else if constexpr (KF == KF_F32_4WF)
        return {reinterpret_cast<const void*>(
                    &igemm_kernel<OP, c.bm, c.bn, c.bk, c.wm, c.wn, 4, true, true>),
                nt};
    else if constexpr (KF == KF_F32_4F)
        return {reinterpret_cast<const void*>(
                    &igemm_kernel<OP, c.bm, c.bn, c.bk, c.wm, c.wn, 4, false, true>),
                nt};
    else if constexpr (KF == KF_F32_4W || KF == KF_F32_1W)
        return {reinterpret_cast<const void*>(
                    &igemm_kernel<OP, c.bm, c.bn, c.bk, c.wm, c.wn, KF == KF_F32_4W ? 4 : 1, true>),
                nt};
    else
        return {reinterpret_cast<const void*>(
                    &igemm_kernel<OP, c.bm, c.bn, c.bk, c.wm, c.wn, KF == KF_F32_4 ? 4 : 1>), nt};
}

template <int OP, int KF>
KernelRef kref_cfg(int cfg) {
    switch (cfg) {
        case 1: return kref<OP, 1, KF>();
        case 2: return kref<OP, 2, KF>();
        case 3: return kref<OP, 3, KF>();
        case 4: return kref<OP, 4, KF>();
        default: return kref<OP, 0, KF>();
    }
}

template <int OP>
KernelRef kref_h16d() {
    if constexpr (OP == OP_WGRAD)
        return {nullptr, 0};
    else
        return {reinterpret_cast<const void*>(&igemm_h16d_kernel<OP>), 64 * H16D_WAVES};
}

template <int OP>
KernelRef kref_op(int cfg, int kf) {
    if (kf == KF_H16D) return kref_h16d<OP>();
    switch (kf) {
        case KF_F32_4: return kref_cfg<OP, KF_F32_4>(cfg);
        case KF_BF_1: return kref_cfg<OP, KF_BF_1>(cfg);
        case KF_BF_4: return kref_cfg<OP, KF_BF_4>(cfg);
        case KF_H16: return kref_cfg<OP, KF_H16>(cfg);
        case KF_H16K: return kref_cfg<OP, KF_H16K>(cfg);
        case KF_F32_4W: return kref_cfg<OP, KF_F32_4W>(cfg);
        case KF_F32_4F: return kref_cfg<OP, KF_F32_4F>(cfg);
        case KF_F32_4WF: return kref_cfg<OP, KF_F32_4WF>(cfg);
        case KF_F32_1W: return kref_cfg<OP, KF_F32_1W>(cfg);
        default: return kref_cfg<OP, KF_F32_1>(cfg);
    }
}

KernelRef kernel_for(int op, int cfg, int kf) {
    if (op == OP_FWD) return kref_op<OP_FWD>(cfg, kf);
    if (op == OP_DGRAD) return kref_op<OP_DGRAD>(cfg, kf);
    return kref_op<OP_WGRAD>(cfg, kf);
}

// Tile configuration for a contraction of M x N (x Kred): the 128x128 tile
// unless one side is at most 64, where a tile of that width wastes less.  A
// forward or data-gradient contraction with a short reduction (a 1x1
// convolution over at most 512 channels) writes much more than it computes;
// 64x64 tiles give it four times as many workgroups to overlap those writes.
int choose_cfg(int op, long M, long N, long Kred) {
    if (M <= 64 && N <= 64) return 4;
    if (N <= 64) return 1;
    if (M <= 64) return (N % 256 == 0 || N >= 1024) ? 2 : 3;
    if (op != OP_WGRAD && Kred <= 512) return 4;
    return 0;
}

}  // namespace

// The fp32 vector kernels address their operands with 32-bit buffer offsets:
// every operand below 2 GB (else the kernels of one element per load take it).
static bool fits_buffer(const ConvGeo& g) {
    const long lim = (1L << 31) - 16;
    return (long)g.N * g.H * g.W * g.C * 4 < lim && (long)g.N * g.P * g.Q * g.K * 4 < lim &&
           (long)g.K * g.R * g.S * g.C * 4 < lim;
}

GemmPlan plan_gemm(int op, const ConvGeo& g, int bf16, int num_cus, int bias_col, int allow_h16d) {
    GemmPlan p{};
    p.op = op;
    p.bf16 = bf16;
    p.bias_col = (op == OP_WGRAD) ? bias_col : 0;
    if (op == OP_FWD) {
        p.M = (long)g.N * g.P * g.Q; p.Ncols = g.K; p.Kred = (long)g.R * g.S * g.C;
    } else if (op == OP_DGRAD) {
        p.M = (long)g.N * g.H * g.W; p.Ncols = g.C; p.Kred = (long)g.R * g.S * g.K;
    } else {
        p.M = g.K; p.Ncols = (long)g.R * g.S * g.C + (p.bias_col ? 1 : 0);
        p.Kred = (long)g.N * g.P * g.Q;
    }
    const bool v4 = ((op == OP_FWD) ? (g.C % 4 == 0) : (g.C % 4 == 0 && g.K % 4 == 0)) &&
                    fits_buffer(g);
    // the FAST fp32 kernels (the k tile is 16 in every fp32 configuration)
    static_assert(kCfgs[0].bk == 16 && kCfgs[1].bk == 16 && kCfgs[2].bk == 16 &&
                      kCfgs[3].bk == 16 && kCfgs[4].bk == 16,
                  "fp32 k tile");
    // (forward and data gradient: at most 7 x 7 taps, which their tap stepping assumes)
    const bool taps7 = g.R <= 7 && g.S <= 7;
    const bool fast32 = (op == OP_FWD && g.C % 16 == 0 && taps7) ||
                        (op == OP_DGRAD && g.st == 1 && g.K % 16 == 0 && taps7) ||
                        (op == OP_WGRAD && g.Q % 16 == 0);
    // bf16 operands in memory: every contiguous axis a multiple of 8 (16 bytes)
    p.h16 = (bf16 && g.C % 8 == 0 && g.K % 8 == 0) ? 1 : 0;
    p.cfg = choose_cfg(op, p.M, p.Ncols, p.Kred);
    if (p.bias_col) {
        // the bias-gradient column rides along unless it adds more than 10% of
        // tiles (then a separate column sum of dy is cheaper)
        const long wn = p.Ncols - 1;
        const int c0 = choose_cfg(op, p.M, wn, p.Kred);
        const long bn = kCfgs[c0].bn;
        if (c0 != p.cfg || 10 * ((p.Ncols + bn - 1) / bn) > 11 * ((wn + bn - 1) / bn)) {
            p.bias_col = 0;
            p.Ncols = wn;
            p.cfg = c0;
        }
    }
    const TileCfg* cp = &kCfgs[p.cfg];
    long tiles = ((p.M + cp->bm - 1) / cp->bm) * ((p.Ncols + cp->bn - 1) / cp->bn);
    int bk = p.h16 ? cp->bkh : (bf16 ? BKH : cp->bk);
    long ktiles = (p.Kred + bk - 1) / bk;
    // fp32: the wide epilogue where the epilogue weighs: a short reduction
    // (writes much relative to what it computes), or a moderate reduction over
    // so few tiles that it is cut into eight or more chunks (the partial tiles
    // written outweigh occupancy).  Long reductions (the weight gradients of
    // large images) and larger tile counts keep the narrow kernel: its
    // occupancy gives them more resident workgroups and reduction chunks.
    if (!bf16) {
        int occ_n = 0;
        const KernelRef kn = kernel_for(op, p.cfg, v4 ? (fast32 ? KF_F32_4F : KF_F32_4) : KF_F32_1);
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ_n, kn.fn, kn.nt, 0) != hipSuccess ||
            occ_n < 1)
            occ_n = 1;
        p.wide = (p.Kred <= 1024 || (p.Kred <= 32768 && 8 * tiles <= (long)num_cus * occ_n)) ? 1 : 0;
    }
    // buffer-load kernels (32-bit offsets): FWD and stride-1 DGRAD with both
    // operands k-major and one tap per k tile; WGRAD on m-major LDS tiles
    const long lim = (1L << 30) - (1L << 20);         // elements of a bf16 operand (< 2 GB)
    const long x_el = (long)g.N * g.H * g.W * g.C, dy_el = (long)g.N * g.P * g.Q * g.K;
    if (p.h16 && (op == OP_FWD || (op == OP_DGRAD && (g.st == 1 || g.st == 2)))) {
        const long cc = (op == OP_FWD) ? g.C : g.K;
        const long a_el = (op == OP_FWD) ? x_el : dy_el;
        p.h16k = (cc % bk == 0 && a_el < lim && p.Ncols * p.Kred < lim) ? 1 : 0;
    } else if (p.h16 && op == OP_WGRAD && !p.bias_col) {
        p.h16k = (x_el < lim && dy_el < lim) ? 1 : 0;
    }
    // the direct-to-LDS kernel: forward and stride-1 data gradient on bf16
    // operands, at most 32 taps, where it measured faster than the 128 x 128
    // tiles (by about a fifth): at least 512 output columns (a multiple of
    // 128), 64 tiles of 256 rows and a reduction of at least 2304.  With
    // fewer columns or a shorter reduction the 256 x 128 tiles lose: their
    // epilogue weighs more and hides less behind the products of the other
    // workgroup (eight waves per CU, against sixteen for the 128 x 128 tiles).
    p.h16d = 0;
    if (allow_h16d && p.h16k && op != OP_WGRAD && (op == OP_FWD || g.st == 1) &&
        p.Ncols % H16D_BN == 0 && p.Ncols >= 512 && p.M >= 64L * H16D_BM && p.Kred >= 2304 &&
        p.Kred % H16D_BK == 0 && !p.bias_col && g.R * g.S <= 32) {
        p.h16d = 1;
        p.cfg = 5;
        cp = &kCfgs[p.cfg];
        tiles = ((p.M + cp->bm - 1) / cp->bm) * ((p.Ncols + cp->bn - 1) / cp->bn);
        bk = H16D_BK;
        ktiles = (p.Kred + bk - 1) / bk;
    }
    const TileCfg& c = *cp;
    // workgroups resident at once
    KernelRef kr = kernel_for(op, p.cfg,
                              p.h16d ? KF_H16D : p.h16k ? KF_H16K
                                     : p.h16 ? KF_H16
                                             : bf16 ? (v4 ? KF_BF_4 : KF_BF_1)
                                                    : (v4 ? (p.wide ? (fast32 ? KF_F32_4WF : KF_F32_4W)
                                                                    : (fast32 ? KF_F32_4F : KF_F32_4))
                                                          : (p.wide ? KF_F32_1W : KF_F32_1)));
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kr.fn, kr.nt, 0) != hipSuccess || occ < 1)
        occ = 1;
    const long slots = (long)num_cus * occ;
    long tfull = tiles, splits = 1;
    // fp32: the time of `cut` tiles each cut into s chunks, in k tiles of a
    // workgroup that shares its CU.  The most loaded CU runs ceil(cut s /
    // CUs) workgroups, occ at a time; a last, partial round takes max(its
    // share, 0.65) of a full one (a lone workgroup gets more than half of the
    // CU's matrix cores); each workgroup adds about 2 k tiles of prologue and
    // epilogue; and each partial tile, written and re-read (8 bytes per
    // output at about 4 TB/s over the device, against 2 BK flops per output
    // at about 75 % of a CU's MFMA rate shared by occ workgroups), costs
    // 0.0288 / occ k tiles.  Measured against the rules it replaced (cut to
    // fill one or two rounds where every tile is cut; the round count of
    // the bf16 rule below otherwise): VGG-19 +1.7 %, the ResNet-152 middle
    // stage +1.9 %, VGG-19 stage 1 +0.6 % (the 14 x 14 layers of VGG-19 take
    // five chunks instead of four: 1.96 rounds instead of 1.53).
    auto f32_cost = [&](long cut, long s) {
        const long wgs = cut * s, n = (wgs + num_cus - 1) / num_cus;
        const long full = n / occ, part = n - full * occ;
        const double r = (double)full + (part ? std::max(0.65, (double)part / occ) : 0.0);
        return r * ((double)ktiles / s + 2.0) + (s > 1 ? (double)wgs * 0.0288 / occ : 0.0);
    };
    auto f32_cut = [&](long cut, long smax) {
        double best = f32_cost(cut, 1);
        long sb = 1;
        for (long s = 2; s <= smax; ++s) {
            const double t = f32_cost(cut, s);
            if (t < best) { best = t; sb = s; }
        }
        return sb;
    };
    if (tiles >= slots) {
        // whole rounds of whole tiles; the tiles of a partial last round cut
        // into s chunks when that shortens it (chunks of at least 4 k tiles)
        const long rounds = tiles / slots, rem = tiles - rounds * slots;
        if (bf16) {
            // time ~ ceil(rem*s/slots)/s; writing and re-reading the partial
            // tile of each chunk (8 bytes per output at about 5 TB/s over the
            // whole device) is weighed against the round it shortens (2 Kred
            // flops per output at about 60% of one CU's MFMA rate), about
            // 4.7 / Kred rounds per chunk (measured: VGG-19 in bf16 +1 %,
            // ResNet-152 +0.3 % against no such term)
            const double pc = 4.7 / (double)p.Kred;
            double best = 1.0;
            for (long s = 2; rem && s <= 16 && s * 4 <= ktiles; ++s) {
                double t = (double)((rem * s + slots - 1) / slots) / s + 0.01 * s + pc * rem * s;
                if (t < best) { best = t; splits = s; }
            }
        } else if (rem) {
            splits = f32_cut(rem, std::min<long>(16, ktiles / 4));
        }
        if (splits > 1) tfull = rounds * slots;
    } else if (bf16) {
        // too few tiles: cut every tile so that one round is filled, each
        // chunk keeping at least 16 k tiles (with fewer, the partial tiles'
        // writes and their reduction cost ResNet-152 3 %)
        splits = std::min<long>(slots / tiles, ktiles / 16);
        if (splits >= 2) tfull = 0;
        else splits = 1;
    } else {
        // fp32, too few tiles: every tile cut, chunks of at least 8 k tiles
        splits = f32_cut(tiles, std::min<long>(ktiles / 8, 4 * slots / tiles + 16));
        if (splits >= 2) tfull = 0;
    }
    long chunk_tiles = (ktiles + splits - 1) / splits;
    p.splits = (int)((ktiles + chunk_tiles - 1) / chunk_tiles);
    // fp32 weight gradient of a fully connected layer over at most 32 images:
    // fcw_kernel, whole FCW_BM x FCW_BN tiles, two workgroups per CU
    // fp32 forward of a fully connected layer over at most 32 images:
    // fcf_kernel, FCF_BN-column tiles each cut into chunks of whole 128-wide k
    // steps, about two workgroups per CU
    p.fcf = 0;
    if (!bf16 && op == OP_FWD && g.H == 1 && g.W == 1 && g.R == 1 && g.S == 1 && p.M <= 32 &&
        g.C % 4 == 0 && fits_buffer(g)) {
        const long tn = (p.Ncols + FCF_BN - 1) / FCF_BN;
        const long kst = (p.Kred + FCF_KSTEP - 1) / FCF_KSTEP;
        long sp = std::max<long>(1, std::min<long>(kst, (2L * num_cus + tn - 1) / tn));
        const long per = (kst + sp - 1) / sp;
        sp = (kst + per - 1) / per;
        p.fcf = 1;
        p.fcw = 0;
        p.cfg = 0;
        p.splits = (int)sp;
        p.kchunk = (int)(per * FCF_KSTEP);
        p.tfull = 0;
        p.nwg = (int)(tn * sp);
        p.ws_floats = (size_t)(tn * sp) * 32 * FCF_BN;
        p.bm = 32;
        p.bn = FCF_BN;
        return p;
    }
    p.fcw = 0;
    if (!bf16 && op == OP_WGRAD && g.H == 1 && g.W == 1 && g.R == 1 && g.S == 1 &&
        p.Kred <= FCW_KMAX && g.C % 4 == 0 && g.K % 4 == 0 && fits_buffer(g)) {
        const long tm = (p.M + FCW_BM - 1) / FCW_BM;
        const long tn = (p.Ncols - p.bias_col + FCW_BN - 1) / FCW_BN;
        p.fcw = 1;
        p.cfg = 0;
        p.splits = 1;
        p.kchunk = (int)p.Kred;
        p.tfull = (int)(((p.M + kCfgs[0].bm - 1) / kCfgs[0].bm) *
                        ((p.Ncols + kCfgs[0].bn - 1) / kCfgs[0].bn));
        p.nwg = (int)std::min<long>(tm * tn, 2L * num_cus);
        p.ws_floats = 0;
        p.bm = FCW_BM;
        p.bn = FCW_BN;
        return p;
    }
    p.kchunk = (int)(chunk_tiles * bk);
    p.tfull = (int)(p.splits > 1 ? tfull : tiles);
    p.nwg = (int)(p.tfull + (tiles - p.tfull) * p.splits);
    p.ws_floats = (size_t)(tiles - p.tfull) * p.splits * c.bm * c.bn;
    p.bm = c.bm;
    p.bn = c.bn;
    return p;
}

namespace {
// Division by a constant d >= 1 for numerators below 2^31 (Granlund and
// Montgomery, round-up method): with l = ceil(log2 d) and m = ceil(2^(31+l)/d),
// m d - 2^(31+l) < d <= 2^l, hence floor(i m / 2^(31+l)) = floor(i / d).
void div_magic(int d, unsigned* m, int* sh) {
    int l = 0;
    while ((1L << l) < d) ++l;
    const unsigned long long num = 1ULL << (31 + l);
    *m = (unsigned)((num + (unsigned long long)d - 1) / (unsigned long long)d);
    *sh = 31 + l;
}
}  // namespace

bool plan_stats(const GemmPlan& plan, int flags) {
    return (flags & ~EPI_BIAS) == 0 && (plan.bf16 || plan.wide) && !plan.h16d && !plan.fcf &&
           !plan.fcw;
}

hipError_t launch_gemm(const GemmPlan& plan, const ConvGeo& g, const float* a, const float* b,
                       float* out, const Epilogue& ep, float* ws, hipStream_t s,
                       const uint16_t* a16, const uint16_t* b16, const uint16_t* b16t) {
    KArgs k{};
    k.g = g;
    k.a = a;
    k.b = b;
    k.out = out;
    k.bias = ep.bias;
    k.mask = ep.mask;
    k.bias_out = ep.bias_out;
    // column statistics: kernels with the wide epilogue only (bf16, or the fp32
    // wide variant); the caller checks plan_stats() before relying on them
    k.stats = plan_stats(plan, ep.flags) ? ep.stats : nullptr;
    k.epi = ep.flags | (plan.bias_col ? EPI_BIASCOL : 0);
    k.M = plan.M;
    k.Ncols = plan.Ncols;
    k.Kred = plan.Kred;
    k.tfull = plan.tfull;
    k.splits = plan.splits;
    k.kchunk = plan.kchunk;
    k.ws = ws;
    k.a16 = a16;
    k.b16 = b16;
    // the bf16 copy: not with a bias-gradient column or column statistics (a
    // batch norm, not a contraction, reads such an output), 16-byte aligned
    if (ep.out16) {
        if (plan.bias_col || k.stats || (((uintptr_t)ep.out16) & 15) != 0)
            return hipErrorInvalidValue;
        k.out16 = reinterpret_cast<unsigned short*>(ep.out16);
    }
    const TileCfg& c = kCfgs[plan.cfg];
    k.tiles_m = (int)((plan.M + c.bm - 1) / c.bm);
    k.tiles_n = (int)((plan.Ncols + c.bn - 1) / c.bn);
    // vector width 4 needs the contiguous axes to be multiples of 4 and the
    // operand bases 16-byte aligned
    bool v4 = (plan.op == OP_FWD) ? (g.C % 4 == 0) : (g.C % 4 == 0 && g.K % 4 == 0);
    v4 = v4 && fits_buffer(g) && ((((uintptr_t)a) | ((uintptr_t)b)) & 15) == 0;
    const bool taps7 = g.R <= 7 && g.S <= 7;
    const bool fast32 = (plan.op == OP_FWD && g.C % 16 == 0 && taps7) ||
                        (plan.op == OP_DGRAD && g.st == 1 && g.K % 16 == 0 && taps7) ||
                        (plan.op == OP_WGRAD && g.Q % 16 == 0);
    // DGRAD on k-major operands takes the transposed weights b16t
    const uint16_t* bk16 = plan.op == OP_DGRAD ? b16t : b16;
    if (plan.op == OP_WGRAD) {
        div_magic(g.Q, &k.mq, &k.sq);
        div_magic(g.P, &k.mp, &k.sp);
    }
    const bool h16k = plan.h16k && a16 && bk16 && ((((uintptr_t)a16) | ((uintptr_t)bk16)) & 15) == 0;
    const bool h16 = !h16k && plan.h16 && plan.bf16 && !plan.bias_col && a16 && b16 &&
                     ((((uintptr_t)a16) | ((uintptr_t)b16)) & 15) == 0;
    if (h16k) k.b16 = bk16;
    const int kf = (h16k && plan.h16d) ? KF_H16D : h16k ? KF_H16K
                        : h16 ? KF_H16
                              : plan.bf16 ? (v4 ? KF_BF_4 : KF_BF_1)
                                          : (v4 ? (plan.wide ? (fast32 ? KF_F32_4WF : KF_F32_4W)
                                                            : (fast32 ? KF_F32_4F : KF_F32_4))
                                                : (plan.wide ? KF_F32_1W : KF_F32_1));
    if (plan.fcf) {
        if (!v4) return hipErrorInvalidValue;
        k.tiles_m = 1;
        k.tiles_n = (int)((plan.Ncols + FCF_BN - 1) / FCF_BN);
        k.tfull = 0;
        hipLaunchKernelGGL(fcf_kernel, dim3(plan.nwg), dim3(256), 0, s, k);
        if (plan.splits <= SK_LANES) {
            const long total = (long)k.tiles_n * 32 * FCF_BN / 4;
            const int blocks = (int)std::min<long>((total + 255) / 256, 16384);
            hipLaunchKernelGGL(igemm_cut_reduce_kernel, dim3(blocks), dim3(256), 0, s, k, 32,
                               FCF_BN);
        } else {
            hipLaunchKernelGGL(igemm_splitk_reduce_kernel, dim3(k.tiles_n * (32 * FCF_BN / SK_EL)),
                               dim3(SK_EL * SK_LANES), 0, s, k, 32, FCF_BN);
        }
        return hipGetLastError();
    }
    if (plan.fcw) {
        if (!v4) return hipErrorInvalidValue;
        k.tiles_m = (int)((plan.M + FCW_BM - 1) / FCW_BM);
        hipLaunchKernelGGL(fcw_kernel, dim3(plan.nwg), dim3(256), 0, s, k);
        return hipGetLastError();
    }
    KernelRef kr = kernel_for(plan.op, plan.cfg, kf);
    void* kargs[] = {&k};
    hipError_t e = hipLaunchKernel(kr.fn, dim3(plan.nwg), dim3(kr.nt), kargs, 0, s);
    const int cut = k.tiles_m * k.tiles_n - plan.tfull;
    if (e != hipSuccess || cut == 0) return e;
    if (k.stats) {
        hipLaunchKernelGGL(igemm_cut_reduce_stats_kernel, dim3(cut), dim3(CRS_THREADS), 0, s, k,
                           c.bm, c.bn);
    } else if (plan.splits <= SK_LANES) {
        const long total = (long)cut * c.bm * c.bn / 4;
        const int blocks = (int)std::min<long>((total + 255) / 256, 16384);
        hipLaunchKernelGGL(igemm_cut_reduce_kernel, dim3(blocks), dim3(256), 0, s, k, c.bm, c.bn);
    } else {
        hipLaunchKernelGGL(igemm_splitk_reduce_kernel, dim3(cut * (c.bm * c.bn / SK_EL)),
                           dim3(SK_EL * SK_LANES), 0, s, k, c.bm, c.bn);
    }
    return hipGetLastError();
}

}  // namespace hp
