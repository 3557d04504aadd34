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
#include <algorithm>
#include <initializer_list>

#include "kernels.h"

namespace hp {
namespace {

constexpr int EW_THREADS = 256;

inline bool aligned16(std::initializer_list<const void*> ptrs) {
    for (const void* q : ptrs)
        if (((uintptr_t)q) & 15) return false;
    return true;
}

inline int ew_blocks(size_t n) {
    size_t b = (n + EW_THREADS - 1) / EW_THREADS;
    return (int)(b < 16384 ? (b ? b : 1) : 16384);
}

// ---- vector helpers: VEC consecutive floats (float4 when VEC == 4) ---------
template <int VEC>
__device__ __forceinline__ void ldv(const float* p, float* o) {
    if constexpr (VEC == 4) {
        const float4 t = *reinterpret_cast<const float4*>(p);
        o[0] = t.x; o[1] = t.y; o[2] = t.z; o[3] = t.w;
    } else {
        o[0] = *p;
    }
}

template <int VEC>
__device__ __forceinline__ void stv(float* p, const float* v) {
    if constexpr (VEC == 4) {
        *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
        *p = v[0];
    }
}

// bf16 copy, round to nearest even (the operand rounding of the bf16 contractions)
__device__ __forceinline__ unsigned bf16_bits(float x) {
    const unsigned u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// VEC values as bf16 to p (8-byte store when VEC == 4)
template <int VEC>
__device__ __forceinline__ void st16v(uint16_t* p, const float* v) {
    if constexpr (VEC == 4) {
        *reinterpret_cast<uint2*>(p) = make_uint2(bf16_bits(v[0]) | (bf16_bits(v[1]) << 16),
                                                  bf16_bits(v[2]) | (bf16_bits(v[3]) << 16));
    } else {
        *p = (uint16_t)bf16_bits(v[0]);
    }
}

__global__ void relu_fwd_kernel(const float* __restrict__ x, float* __restrict__ y, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        y[i] = fmaxf(x[i], 0.f);
}

template <int VEC>
__global__ void relu_bwd_kernel(const float* __restrict__ y, const float* __restrict__ dy,
                                float* __restrict__ dx, size_t n, int acc) {
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < n;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        float yv[VEC], g[VEC], d[VEC];
        ldv<VEC>(y + i, yv);
        ldv<VEC>(dy + i, g);
        if (acc) ldv<VEC>(dx + i, d);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const float v = yv[j] > 0.f ? g[j] : 0.f;
            d[j] = acc ? d[j] + v : v;
        }
        stv<VEC>(dx + i, d);
    }
}

template <int VEC>
__global__ void add_fwd_kernel(const float* __restrict__ a, const float* __restrict__ b,
                               float* __restrict__ y, size_t n, int relu,
                               uint16_t* __restrict__ y16) {
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < n;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        float av[VEC], bv[VEC];
        ldv<VEC>(a + i, av);
        ldv<VEC>(b + i, bv);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const float v = av[j] + bv[j];
            av[j] = relu ? fmaxf(v, 0.f) : v;
        }
        stv<VEC>(y + i, av);
        if (y16) st16v<VEC>(y16 + i, av);
    }
}

template <int VEC>
__global__ void copy_or_acc_kernel(const float* __restrict__ v, float* __restrict__ out, size_t n,
                                   int acc) {
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < n;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        float a[VEC], o[VEC];
        ldv<VEC>(v + i, a);
        if (acc) {
            ldv<VEC>(out + i, o);
#pragma unroll
            for (int j = 0; j < VEC; ++j) a[j] = o[j] + a[j];
        }
        stv<VEC>(out + i, a);
    }
}

// max-pool forward: padded taps never win; the first maximum in row-major
// window order is kept (strict '>' comparison).
// max-pool forward: VEC consecutive channels of one output pixel per thread
// arg (optional): the window tap r * S + s of the first maximum, one byte per
// output element (255: none), for the backward pass of overlapping windows.
template <int VEC>
__global__ void maxpool_fwd_kernel(const float* __restrict__ x, float* __restrict__ y, int N, int H,
                                   int W, int C, int R, int S, int st, int pad, int P, int Q,
                                   uint16_t* __restrict__ y16, uint8_t* __restrict__ arg) {
    const size_t total = (size_t)N * P * Q * C;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < total;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        const int c = (int)(i % C);
        size_t t = i / C;
        const int q = (int)(t % Q); t /= Q;
        const int p = (int)(t % P);
        const int n = (int)(t / P);
        float m[VEC];
        int best[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) best[j] = 255;     // no tap (a window of padding)
        bool any = false;
        for (int r = 0; r < R; ++r) {
            const int h = p * st - pad + r;
            if (h < 0 || h >= H) continue;
            for (int s = 0; s < S; ++s) {
                const int w = q * st - pad + s;
                if (w < 0 || w >= W) continue;
                float v[VEC];
                ldv<VEC>(x + (((size_t)n * H + h) * W + w) * C + c, v);
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    if (!any || v[j] > m[j]) { m[j] = v[j]; best[j] = r * S + s; }
                any = true;
            }
        }
        stv<VEC>(y + i, m);
        if (y16) st16v<VEC>(y16 + i, m);
        if (arg) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) arg[i + j] = (uint8_t)best[j];
        }
    }
}

// max-pool backward as a gather: each input element sums dy over the windows
// whose first maximum it is (the window's argmax is recomputed from x), in
// window order; VEC consecutive channels per thread.
template <int VEC>
__global__ void maxpool_bwd_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                   float* __restrict__ dx, int N, int H, int W, int C, int R,
                                   int S, int st, int pad, int P, int Q, int acc,
                                   const float* __restrict__ mask, uint16_t* __restrict__ dx16) {
    const size_t total = (size_t)N * H * W * C;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < total;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        const int c = (int)(i % C);
        size_t t = i / C;
        const int w0 = (int)(t % W); t /= W;
        const int h0 = (int)(t % H);
        const int n = (int)(t / H);
        float sum[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) sum[j] = 0.f;
        for (int r = 0; r < R; ++r) {
            const int tp = h0 + pad - r;
            if (tp < 0 || tp % st) continue;
            const int p = tp / st;
            if (p >= P) continue;
            for (int s = 0; s < S; ++s) {
                const int tq = w0 + pad - s;
                if (tq < 0 || tq % st) continue;
                const int q = tq / st;
                if (q >= Q) continue;
                // first argmax of window (p, q), per channel
                int best[VEC];
                float m[VEC];
#pragma unroll
                for (int j = 0; j < VEC; ++j) { best[j] = -1; m[j] = 0.f; }
                for (int rr = 0; rr < R; ++rr) {
                    const int h = p * st - pad + rr;
                    if (h < 0 || h >= H) continue;
                    for (int ss = 0; ss < S; ++ss) {
                        const int w = q * st - pad + ss;
                        if (w < 0 || w >= W) continue;
                        float v[VEC];
                        ldv<VEC>(x + (((size_t)n * H + h) * W + w) * C + c, v);
#pragma unroll
                        for (int j = 0; j < VEC; ++j)
                            if (best[j] < 0 || v[j] > m[j]) { m[j] = v[j]; best[j] = rr * S + ss; }
                    }
                }
                float g[VEC];
                ldv<VEC>(dy + (((size_t)n * P + p) * Q + q) * C + c, g);
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    if (best[j] == r * S + s) sum[j] += g[j];
            }
        }
        if (mask) {
            float mk[VEC];
            ldv<VEC>(mask + i, mk);
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (!(mk[j] > 0.f)) sum[j] = 0.f;
        }
        if (acc) {
            float d[VEC];
            ldv<VEC>(dx + i, d);
#pragma unroll
            for (int j = 0; j < VEC; ++j) sum[j] = d[j] + sum[j];
        }
        stv<VEC>(dx + i, sum);
        if (dx16) st16v<VEC>(dx16 + i, sum);
    }
}

// max-pool backward as a gather with the taps the forward pass recorded:
// each input element sums dy over the windows whose first maximum it is, in
// window order, reading one byte per candidate window instead of the window.
template <int VEC>
__global__ void maxpool_bwd_arg_kernel(const uint8_t* __restrict__ arg,
                                       const float* __restrict__ dy, float* __restrict__ dx,
                                       int N, int H, int W, int C, int R, int S, int st, int pad,
                                       int P, int Q, int acc, const float* __restrict__ mask,
                                       uint16_t* __restrict__ dx16) {
    const size_t total = (size_t)N * H * W * C;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < total;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        const int c = (int)(i % C);
        size_t t = i / C;
        const int w0 = (int)(t % W); t /= W;
        const int h0 = (int)(t % H);
        const int n = (int)(t / H);
        float sum[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) sum[j] = 0.f;
        for (int r = 0; r < R; ++r) {
            const int tp = h0 + pad - r;
            if (tp < 0 || tp % st) continue;
            const int p = tp / st;
            if (p >= P) continue;
            for (int s = 0; s < S; ++s) {
                const int tq = w0 + pad - s;
                if (tq < 0 || tq % st) continue;
                const int q = tq / st;
                if (q >= Q) continue;
                const size_t o = (((size_t)n * P + p) * Q + q) * C + c;
                float g[VEC];
                ldv<VEC>(dy + o, g);
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    if (arg[o + j] == r * S + s) sum[j] += g[j];
            }
        }
        if (mask) {
            float mk[VEC];
            ldv<VEC>(mask + i, mk);
#pragma unroll
            for (int j = 0; j < VEC; ++j)
                if (!(mk[j] > 0.f)) sum[j] = 0.f;
        }
        if (acc) {
            float d[VEC];
            ldv<VEC>(dx + i, d);
#pragma unroll
            for (int j = 0; j < VEC; ++j) sum[j] = d[j] + sum[j];
        }
        stv<VEC>(dx + i, sum);
        if (dx16) st16v<VEC>(dx16 + i, sum);
    }
}

// max-pool backward for non-overlapping windows (window = stride, no padding,
// windows tile the input exactly): one thread per output pixel and VEC
// channels writes its whole window (dy at the first argmax, zero elsewhere).
// RT > 0 fixes the window edge at compile time and keeps the taps in
// registers; when the pooled input is a ReLU output the taps are the mask.
template <int RT, int VEC>
__global__ void maxpool_bwd_tiled_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                         float* __restrict__ dx, int N, int H, int W, int C, int Rr,
                                         int P, int Q, int acc, const float* __restrict__ mask,
                                       uint16_t* __restrict__ dx16) {
    const int R = RT > 0 ? RT : Rr;
    const size_t total = (size_t)N * P * Q * C;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < total;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        const int c = (int)(i % C);
        size_t t = i / C;
        const int q = (int)(t % Q); t /= Q;
        const int p = (int)(t % P);
        const int n = (int)(t / P);
        const size_t base = (((size_t)n * H + p * R) * W + q * R) * C + c;
        float g[VEC];
        ldv<VEC>(dy + i, g);
        if constexpr (RT > 0) {
            float v[RT * RT][VEC];
            float m[VEC];
            int best[VEC];
#pragma unroll
            for (int k = 0; k < RT * RT; ++k) {
                ldv<VEC>(x + base + ((size_t)(k / RT) * W + k % RT) * C, v[k]);
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    if (k == 0 || v[k][j] > m[j]) { m[j] = v[k][j]; best[j] = k; }
            }
#pragma unroll
            for (int k = 0; k < RT * RT; ++k) {
                const size_t e = base + ((size_t)(k / RT) * W + k % RT) * C;
                float o[VEC], mk[VEC], d[VEC];
                if (mask && mask != x) ldv<VEC>(mask + e, mk);
                if (acc) ldv<VEC>(dx + e, d);
#pragma unroll
                for (int j = 0; j < VEC; ++j) {
                    o[j] = (k == best[j]) ? g[j] : 0.f;
                    if (mask && !((mask == x ? v[k][j] : mk[j]) > 0.f)) o[j] = 0.f;
                    if (acc) o[j] = d[j] + o[j];
                }
                stv<VEC>(dx + e, o);
                if (dx16) st16v<VEC>(dx16 + e, o);
            }
        } else {
            float m[VEC];
            int best[VEC];
            for (int k = 0; k < R * R; ++k) {
                float v[VEC];
                ldv<VEC>(x + base + ((size_t)(k / R) * W + k % R) * C, v);
#pragma unroll
                for (int j = 0; j < VEC; ++j)
                    if (k == 0 || v[j] > m[j]) { m[j] = v[j]; best[j] = k; }
            }
            for (int k = 0; k < R * R; ++k) {
                const size_t e = base + ((size_t)(k / R) * W + k % R) * C;
                float o[VEC], mk[VEC], d[VEC];
                if (mask) ldv<VEC>(mask + e, mk);
                if (acc) ldv<VEC>(dx + e, d);
#pragma unroll
                for (int j = 0; j < VEC; ++j) {
                    o[j] = (k == best[j]) ? g[j] : 0.f;
                    if (mask && !(mk[j] > 0.f)) o[j] = 0.f;
                    if (acc) o[j] = d[j] + o[j];
                }
                stv<VEC>(dx + e, o);
                if (dx16) st16v<VEC>(dx16 + e, o);
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
// Partials: workgroup (bx, by) reduces rows [by*rb, by*rb + rb) of a strip of
// channels.  256 threads = cg channel lanes (VEC consecutive channels each,
// one vector load per row) x 256/cg row lanes; a thread visits its rows four
// at a time (independent loads in flight) and the row lanes are combined in
// LDS in a fixed order.  rb is chosen so that the grid has a few hundred
// workgroups whatever the shape (few rows x many channels or the reverse).
//
// MODE_SUM:     part0 = sum v
// MODE_MOMENTS: part0 = mean of the block's rows, part1 = sum of squared
//               deviations from it (one pass: each thread sums deviations from
//               its first value, then the thread and block statistics are
//               merged with the pairwise update of Chan, Golub and LeVeque)
// MODE_BNBWD:   part0 = sum g, part1 = sum g * xhat, g = v masked by relu_y > 0
//               when relu_y is given, xhat = (x - mean) * invstd
enum { MODE_SUM = 0, MODE_MOMENTS = 1, MODE_BNBWD = 2 };
constexpr int CS_THREADS = 256;


// (n_a, mean_a, m2_a) <- merge with (n_b, mean_b, m2_b)
__device__ __forceinline__ void chan_merge(float& na, float& mean_a, float& m2a, float nb,
                                           float mean_b, float m2b) {
    const float n = na + nb;
    if (nb == 0.f) return;
    if (na == 0.f) { na = nb; mean_a = mean_b; m2a = m2b; return; }
    const float d = mean_b - mean_a;
    const float f = nb / n;
    mean_a = mean_a + d * f;
    m2a = (m2a + m2b) + d * d * (na * f);
    na = n;
}

template <int MODE, int VEC>
__global__ void __launch_bounds__(CS_THREADS)
colsum_partial_kernel(const float* __restrict__ v, const float* __restrict__ x,
                      const float* __restrict__ relu_y, const float* __restrict__ mean,
                      const float* __restrict__ invstd, long M, int C, int cg, long rb,
                      float* __restrict__ part0, float* __restrict__ part1) {
    __shared__ float red0[CS_THREADS * VEC];
    __shared__ float red1[CS_THREADS * VEC];
    __shared__ float cnt[CS_THREADS];
    const int cl = threadIdx.x % cg;
    const int rl = threadIdx.x / cg;
    const int RL = CS_THREADS / cg;
    const int c0 = (blockIdx.x * cg + cl) * VEC;
    const bool on = c0 < C;
    const long r0 = (long)blockIdx.y * rb;
    const long r1 = min(r0 + rb, M);
    float a0[VEC], a1[VEC], k[VEC], mu[VEC], is[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) a0[j] = a1[j] = k[j] = mu[j] = is[j] = 0.f;
    int n = 0;
    auto acc = [&](const float* t, const float* xx, const float* yy) {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            if constexpr (MODE == MODE_SUM) {
                a0[j] += t[j];
            } else if constexpr (MODE == MODE_MOMENTS) {
                const float d = t[j] - k[j];
                a0[j] += d;
                a1[j] += d * d;
            } else {
                const float g = (relu_y && !(yy[j] > 0.f)) ? 0.f : t[j];
                const float xh = (xx[j] - mu[j]) * is[j];
                a0[j] += g;
                a1[j] += g * xh;
            }
        }
    };
    if (on) {
        if constexpr (MODE == MODE_BNBWD) {
            ldv<VEC>(mean + c0, mu);
            ldv<VEC>(invstd + c0, is);
        }
        long r = r0 + rl;
        if constexpr (MODE == MODE_MOMENTS) {
            if (r < r1) ldv<VEC>(v + (size_t)r * C + c0, k);
        }
        for (; r + 3L * RL < r1; r += 4L * RL) {
            float t[4][VEC], xx[4][VEC], yy[4][VEC];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const size_t idx = (size_t)(r + (long)u * RL) * C + c0;
                ldv<VEC>(v + idx, t[u]);
                if constexpr (MODE == MODE_BNBWD) {
                    ldv<VEC>(x + idx, xx[u]);
                    if (relu_y) ldv<VEC>(relu_y + idx, yy[u]);
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) acc(t[u], xx[u], yy[u]);
            n += 4;
        }
        for (; r < r1; r += RL) {
            float t[VEC], xx[VEC], yy[VEC];
            const size_t idx = (size_t)r * C + c0;
            ldv<VEC>(v + idx, t);
            if constexpr (MODE == MODE_BNBWD) {
                ldv<VEC>(x + idx, xx);
                if (relu_y) ldv<VEC>(relu_y + idx, yy);
            }
            acc(t, xx, yy);
            n += 1;
        }
    }
    if constexpr (MODE == MODE_MOMENTS) {
        // thread statistics: mean = shift + mean deviation
        const float fn = (float)n;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            if (n > 0) {
                const float md = a0[j] / fn;
                a1[j] = fmaxf(a1[j] - a0[j] * md, 0.f);
                a0[j] = k[j] + md;
            }
        }
        cnt[threadIdx.x] = fn;
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        red0[threadIdx.x * VEC + j] = a0[j];
        red1[threadIdx.x * VEC + j] = a1[j];
    }
    __syncthreads();
    if (rl == 0 && on) {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            float s0 = red0[cl * VEC + j], s1 = red1[cl * VEC + j];
            float na = (MODE == MODE_MOMENTS) ? cnt[cl] : 0.f;
            for (int l = 1; l < RL; ++l) {
                const int th = l * cg + cl;
                if constexpr (MODE == MODE_MOMENTS) {
                    chan_merge(na, s0, s1, cnt[th], red0[th * VEC + j], red1[th * VEC + j]);
                } else {
                    s0 += red0[th * VEC + j];
                    s1 += red1[th * VEC + j];
                }
            }
            if (c0 + j < C) {
                part0[(size_t)blockIdx.y * C + c0 + j] = s0;
                if (MODE != MODE_SUM) part1[(size_t)blockIdx.y * C + c0 + j] = s1;
            }
        }
    }
}

// Combination of the nb row-block partials of each channel: workgroup = 8
// channels x 128 lanes; lane l takes blocks l, l+128, ... in order, then the
// lane results are combined by a fixed binary tree (lane l with l + 64, then
// l + 32, ...), so the order of every addition is fixed.
//   FIN_SUM:   out0 = sum part0
//   FIN_SUM2:  out0 = sum part0, out1 = sum part1
//   FIN_STATS: merge (block mean, block squared deviations); out0 = mean,
//              out1 = 1 / sqrt(biased variance + eps)
enum { FIN_SUM = 0, FIN_SUM2 = 1, FIN_STATS = 2 };
constexpr int CF_CH = 8, CF_LANES = 128;    // (16 x 64: ResNet-152 -0.2 %; 4 x 256 no better)

template <int FIN>
__global__ void __launch_bounds__(CF_CH * CF_LANES)
colsum_final_kernel(const float* __restrict__ part0, const float* __restrict__ part1, int nb,
                    long rb, int C, long M, float eps, float* __restrict__ out0,
                    float* __restrict__ out1) {
    __shared__ float r0[CF_LANES][CF_CH], r1[CF_LANES][CF_CH], rn[CF_LANES][CF_CH];
    const int cl = threadIdx.x % CF_CH;
    const int ln = threadIdx.x / CF_CH;
    const int c = blockIdx.x * CF_CH + cl;
    float s0 = 0.f, s1 = 0.f, na = 0.f;
    if (c < C) {
        for (int b = ln; b < nb; b += CF_LANES) {
            const float p0 = part0[(size_t)b * C + c];
            if constexpr (FIN == FIN_STATS) {
                const float cnt = (float)min(rb, M - (long)b * rb);
                chan_merge(na, s0, s1, cnt, p0, part1[(size_t)b * C + c]);
            } else {
                s0 += p0;
                if (FIN == FIN_SUM2) s1 += part1[(size_t)b * C + c];
            }
        }
    }
    r0[ln][cl] = s0;
    r1[ln][cl] = s1;
    rn[ln][cl] = na;
    __syncthreads();
    for (int off = CF_LANES / 2; off > 0; off >>= 1) {
        if (ln < off) {
            if constexpr (FIN == FIN_STATS) {
                float n = rn[ln][cl], m = r0[ln][cl], q = r1[ln][cl];
                chan_merge(n, m, q, rn[ln + off][cl], r0[ln + off][cl], r1[ln + off][cl]);
                rn[ln][cl] = n;
                r0[ln][cl] = m;
                r1[ln][cl] = q;
            } else {
                r0[ln][cl] += r0[ln + off][cl];
                if (FIN == FIN_SUM2) r1[ln][cl] += r1[ln + off][cl];
            }
        }
        __syncthreads();
    }
    if (ln == 0 && c < C) {
        if constexpr (FIN == FIN_STATS) {
            out0[c] = r0[0][cl];
            out1[c] = 1.f / sqrtf(r1[0][cl] / (float)M + eps);
        } else {
            out0[c] = r0[0][cl];
            if (FIN == FIN_SUM2) out1[c] = r1[0][cl];
        }
    }
}

template <int VEC>
__global__ void bn_apply_kernel(const float* __restrict__ x, long M, int C,
                                const float* __restrict__ gamma, const float* __restrict__ beta,
                                const float* __restrict__ mean, const float* __restrict__ invstd,
                                float* __restrict__ y, int relu, uint16_t* __restrict__ y16) {
    const size_t total = (size_t)M * C;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < total;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        const int c = (int)(i % C);
        float xv[VEC], ga[VEC], be[VEC], mu[VEC], is[VEC];
        ldv<VEC>(x + i, xv);
        ldv<VEC>(gamma + c, ga);
        ldv<VEC>(beta + c, be);
        ldv<VEC>(mean + c, mu);
        ldv<VEC>(invstd + c, is);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const float v = ga[j] * ((xv[j] - mu[j]) * is[j]) + be[j];
            xv[j] = relu ? fmaxf(v, 0.f) : v;
        }
        stv<VEC>(y + i, xv);
        if (y16) st16v<VEC>(y16 + i, xv);
    }
}

// dx = gamma*invstd*(dy' - sdy/M - xhat*sdyx/M)
template <int VEC>
__global__ void bn_bwd_apply_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                                    const float* __restrict__ relu_y, long M, int C,
                                    const float* __restrict__ gamma,
                                    const float* __restrict__ mean,
                                    const float* __restrict__ invstd,
                                    const float* __restrict__ sdy, const float* __restrict__ sdyx,
                                    float* __restrict__ dx, int acc,
                                    uint16_t* __restrict__ dx16) {
    const size_t total = (size_t)M * C;
    const float invM = 1.f / (float)M;
    for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC; i < total;
         i += (size_t)gridDim.x * blockDim.x * VEC) {
        const int c = (int)(i % C);
        float g[VEC], xv[VEC], yv[VEC], d[VEC], ga[VEC], mu[VEC], is[VEC], s0[VEC], s1[VEC];
        ldv<VEC>(dy + i, g);
        ldv<VEC>(x + i, xv);
        if (relu_y) ldv<VEC>(relu_y + i, yv);
        if (acc) ldv<VEC>(dx + i, d);
        ldv<VEC>(gamma + c, ga);
        ldv<VEC>(mean + c, mu);
        ldv<VEC>(invstd + c, is);
        ldv<VEC>(sdy + c, s0);
        ldv<VEC>(sdyx + c, s1);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const float gj = (relu_y && !(yv[j] > 0.f)) ? 0.f : g[j];
            const float xh = (xv[j] - mu[j]) * is[j];
            const float v = ga[j] * is[j] * (gj - s0[j] * invM - xh * (s1[j] * invM));
            d[j] = acc ? d[j] + v : v;
        }
        stv<VEC>(dx + i, d);
        if (dx16) st16v<VEC>(dx16 + i, d);
    }
}


__global__ void cast_bf16_kernel(const float* __restrict__ src, uint16_t* __restrict__ dst,
                                 size_t n, int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const float4* s4 = reinterpret_cast<const float4*>(src);
    uint2* d2 = reinterpret_cast<uint2*>(dst);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        const float4 v = s4[i];
        d2[i] = make_uint2(bf16_bits(v.x) | (bf16_bits(v.y) << 16),
                           bf16_bits(v.z) | (bf16_bits(v.w) << 16));
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = (uint16_t)bf16_bits(src[i]);
}

// Channel padding of a conv whose input channel count is not a multiple of
// the contraction's vector width: dst[r][c] = src[r][c] for c < C, 0 up to Cp
// (fp32, or bf16 rounded to nearest even); and the reverse for the weight
// gradient computed on the padded geometry.
__global__ void pad_channels_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                    uint16_t* __restrict__ dst16, size_t rows, int C, int Cp) {
    const size_t n = rows * (size_t)Cp;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        const size_t r = i / Cp;
        const int c = (int)(i - r * Cp);
        const float v = c < C ? src[r * C + c] : 0.f;
        if (dst16) dst16[i] = (uint16_t)bf16_bits(v);
        else dst[i] = v;
    }
}

__global__ void unpad_channels_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                      size_t rows, int C, int Cp) {
    const size_t n = rows * (size_t)C;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        const size_t r = i / C;
        dst[i] = src[r * Cp + (i - r * C)];
    }
}

// Transposed bf16 copies of conv/FC weights for the data gradient:
// dst[off + (c * RS + rs) * K + k] = bf16(src[off + (k * RS + rs) * C + c]) for
// every layer of the table.  A workgroup transposes one 64 (k) x 64 (c) tile
// of one tap through LDS, so that both the reads (along c) and the writes
// (along k) are contiguous; it finds its layer by binary search over the
// layers' first tile numbers.
constexpr int WT_T = WT_TILE;

__global__ void __launch_bounds__(256) cast_bf16_t_kernel(const float* __restrict__ src,
                                                          uint16_t* __restrict__ dst,
                                                          const WtLayer* __restrict__ table,
                                                          int nlayers) {
    __shared__ float tile[WT_T][WT_T + 1];
    const int b = blockIdx.x;
    int lo = 0, hi = nlayers - 1;      // last layer whose first tile is <= b
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (table[mid].tile0 <= b) lo = mid;
        else hi = mid - 1;
    }
    const WtLayer L = table[lo];
    const int tkn = (L.K + WT_T - 1) / WT_T, tcn = (L.C + WT_T - 1) / WT_T;
    int tl = b - L.tile0;
    const int c0 = (tl % tcn) * WT_T;
    tl /= tcn;
    const int k0 = (tl % tkn) * WT_T;
    const int rs = tl / tkn;
    for (int e = threadIdx.x; e < WT_T * WT_T; e += 256) {
        const int kk = e / WT_T, cc = e % WT_T;
        const int k = k0 + kk, c = c0 + cc;
        tile[kk][cc] = (k < L.K && c < L.C) ? src[L.off + ((long)k * L.RS + rs) * L.C + c] : 0.f;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < WT_T * WT_T; e += 256) {
        const int cc = e / WT_T, kk = e % WT_T;
        const int k = k0 + kk, c = c0 + cc;
        if (k < L.K && c < L.C)
            dst[L.off + ((long)c * L.RS + rs) * L.K + k] = (uint16_t)bf16_bits(tile[kk][cc]);
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
    if (n % 4 == 0 && aligned16({y, dy, dx}))
        hipLaunchKernelGGL(relu_bwd_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, y, dy,
                           dx, n, accumulate);
    else
        hipLaunchKernelGGL(relu_bwd_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, y, dy, dx,
                           n, accumulate);
    return hipGetLastError();
}

hipError_t launch_add_fwd(const float* a, const float* b, float* y, size_t n, int relu,
                          hipStream_t s, uint16_t* y16) {
    if (n % 4 == 0 && aligned16({a, b, y}) && ((uintptr_t)y16 & 7) == 0)
        hipLaunchKernelGGL(add_fwd_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, a, b, y,
                           n, relu, y16);
    else
        hipLaunchKernelGGL(add_fwd_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, a, b, y, n,
                           relu, y16);
    return hipGetLastError();
}

hipError_t launch_copy_or_acc(const float* v, float* out, size_t n, int accumulate,
                              hipStream_t s) {
    if (n % 4 == 0 && aligned16({v, out}))
        hipLaunchKernelGGL(copy_or_acc_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, v,
                           out, n, accumulate);
    else
        hipLaunchKernelGGL(copy_or_acc_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, v, out,
                           n, accumulate);
    return hipGetLastError();
}

hipError_t launch_maxpool_fwd(const float* x, float* y, int N, int H, int W, int C, int R, int S,
                              int st, int pad, int P, int Q, hipStream_t s, uint16_t* y16,
                              uint8_t* arg) {
    size_t n = (size_t)N * P * Q * C;
    if (C % 4 == 0 && aligned16({x, y}) && ((uintptr_t)y16 & 7) == 0)
        hipLaunchKernelGGL(maxpool_fwd_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, x,
                           y, N, H, W, C, R, S, st, pad, P, Q, y16, arg);
    else
        hipLaunchKernelGGL(maxpool_fwd_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, y,
                           N, H, W, C, R, S, st, pad, P, Q, y16, arg);
    return hipGetLastError();
}

bool maxpool_tiled(int H, int W, int R, int S, int st, int pad, int P, int Q) {
    return R == S && R == st && pad == 0 && P * st == H && Q * st == W;
}

hipError_t launch_maxpool_bwd(const float* x, const float* dy, float* dx, int N, int H, int W,
                              int C, int R, int S, int st, int pad, int P, int Q, int accumulate,
                              const float* mask, hipStream_t s, const uint8_t* arg, uint16_t* dx16) {
    const bool v4 = C % 4 == 0 && aligned16({x, dy, dx, mask}) && ((uintptr_t)dx16 & 7) == 0;
    if (maxpool_tiled(H, W, R, S, st, pad, P, Q)) {
        size_t n = (size_t)N * P * Q * C;
        const dim3 g(ew_blocks(v4 ? n / 4 : n)), b(EW_THREADS);
        if (R == 2 && v4)
            hipLaunchKernelGGL((maxpool_bwd_tiled_kernel<2, 4>), g, b, 0, s, x, dy, dx, N, H, W, C,
                               R, P, Q, accumulate, mask, dx16);
        else if (R == 2)
            hipLaunchKernelGGL((maxpool_bwd_tiled_kernel<2, 1>), g, b, 0, s, x, dy, dx, N, H, W, C,
                               R, P, Q, accumulate, mask, dx16);
        else if (v4)
            hipLaunchKernelGGL((maxpool_bwd_tiled_kernel<0, 4>), g, b, 0, s, x, dy, dx, N, H, W, C,
                               R, P, Q, accumulate, mask, dx16);
        else
            hipLaunchKernelGGL((maxpool_bwd_tiled_kernel<0, 1>), g, b, 0, s, x, dy, dx, N, H, W, C,
                               R, P, Q, accumulate, mask, dx16);
        return hipGetLastError();
    }
    size_t n = (size_t)N * H * W * C;
    if (arg && v4)
        hipLaunchKernelGGL(maxpool_bwd_arg_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s,
                           arg, dy, dx, N, H, W, C, R, S, st, pad, P, Q, accumulate, mask, dx16);
    else if (arg)
        hipLaunchKernelGGL(maxpool_bwd_arg_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s,
                           arg, dy, dx, N, H, W, C, R, S, st, pad, P, Q, accumulate, mask, dx16);
    else if (v4)
        hipLaunchKernelGGL(maxpool_bwd_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, x,
                           dy, dx, N, H, W, C, R, S, st, pad, P, Q, accumulate, mask, dx16);
    else
        hipLaunchKernelGGL(maxpool_bwd_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, dy,
                           dx, N, H, W, C, R, S, st, pad, P, Q, accumulate, mask, dx16);
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

namespace {

// Launch shape of a column reduction: VEC channels per thread (4 when the
// channel count and the operands allow float4 loads), cg channel lanes, gx x nb
// workgroups of rb rows.
struct ColPlan {
    int vec, cg, gx, nb;
    long rb;
};

ColPlan col_plan(long M, int C, int vec) {
    ColPlan p;
    p.vec = vec;
    const int groups = (C + vec - 1) / vec;
    int cg = 1;
    while (cg < groups && cg < 64) cg <<= 1;
    p.cg = cg;
    const int rl = CS_THREADS / cg;
    p.gx = (groups + cg - 1) / cg;
    const long want = std::max(1, 512 / p.gx);
    const long most = std::max(1L, (M + 4L * rl - 1) / (4L * rl));
    const long nb = std::min(want, most);
    long rb = (std::max(M, 1L) + nb - 1) / nb;
    rb = (rb + rl - 1) / rl * rl;
    p.rb = rb;
    p.nb = (int)((std::max(M, 1L) + rb - 1) / rb);
    return p;
}

bool vec4_ok(int C, std::initializer_list<const void*> ptrs) {
    if (C % 4) return false;
    for (const void* q : ptrs)
        if (((uintptr_t)q) & 15) return false;
    return true;
}

int col_blocks_max(long M, int C) {
    return std::max(col_plan(M, C, 4).nb, col_plan(M, C, 1).nb);
}

template <int MODE>
void launch_partial(const ColPlan& p, const float* v, const float* x, const float* relu_y,
                    const float* mean, const float* invstd, long M, int C, float* part0,
                    float* part1, hipStream_t s) {
    const dim3 grid(p.gx, p.nb);
    if (p.vec == 4)
        hipLaunchKernelGGL((colsum_partial_kernel<MODE, 4>), grid, dim3(CS_THREADS), 0, s, v, x,
                           relu_y, mean, invstd, M, C, p.cg, p.rb, part0, part1);
    else
        hipLaunchKernelGGL((colsum_partial_kernel<MODE, 1>), grid, dim3(CS_THREADS), 0, s, v, x,
                           relu_y, mean, invstd, M, C, p.cg, p.rb, part0, part1);
}

template <int FIN>
void launch_final(const ColPlan& p, const float* part0, const float* part1, long M, int C,
                  float eps, float* out0, float* out1, hipStream_t s) {
    hipLaunchKernelGGL((colsum_final_kernel<FIN>), dim3((C + CF_CH - 1) / CF_CH),
                       dim3(CF_CH * CF_LANES), 0, s, part0, part1, p.nb, p.rb, C, M, eps, out0,
                       out1);
}

}  // namespace

size_t colsum_ws_floats(long M, int C) { return (size_t)col_blocks_max(M, C) * C; }

hipError_t launch_colsum(const float* v, long M, int C, float* out, float* ws, hipStream_t s) {
    const ColPlan p = col_plan(M, C, vec4_ok(C, {v}) ? 4 : 1);
    launch_partial<MODE_SUM>(p, v, nullptr, nullptr, nullptr, nullptr, M, C, ws, nullptr, s);
    launch_final<FIN_SUM>(p, ws, nullptr, M, C, 0.f, out, nullptr, s);
    return hipGetLastError();
}

size_t bn_ws_floats(long M, int C) { return 2 * (size_t)col_blocks_max(M, C) * C; }

hipError_t launch_bn_fwd(const float* x, long M, int C, const float* gamma, const float* beta,
                         float eps, float* y, float* mean, float* invstd, int relu, float* ws,
                         hipStream_t s, uint16_t* y16) {
    const ColPlan p = col_plan(M, C, vec4_ok(C, {x}) ? 4 : 1);
    float* p0 = ws;
    float* p1 = ws + (size_t)p.nb * C;
    launch_partial<MODE_MOMENTS>(p, x, nullptr, nullptr, nullptr, nullptr, M, C, p0, p1, s);
    launch_final<FIN_STATS>(p, p0, p1, M, C, eps, mean, invstd, s);
    size_t n = (size_t)M * C;
    if (vec4_ok(C, {x, y, gamma, beta, mean, invstd}) && ((uintptr_t)y16 & 7) == 0)
        hipLaunchKernelGGL(bn_apply_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, x, M,
                           C, gamma, beta, mean, invstd, y, relu, y16);
    else
        hipLaunchKernelGGL(bn_apply_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, M, C,
                           gamma, beta, mean, invstd, y, relu, y16);
    return hipGetLastError();
}

hipError_t launch_bn_fwd_partials(const float* x, long M, int C, const float* gamma,
                                  const float* beta, float eps, float* y, float* mean,
                                  float* invstd, int relu, const float* part0, const float* part1,
                                  int nb, long rb, hipStream_t s, uint16_t* y16) {
    ColPlan p{};
    p.nb = nb;
    p.rb = rb;
    launch_final<FIN_STATS>(p, part0, part1, M, C, eps, mean, invstd, s);
    size_t n = (size_t)M * C;
    if (vec4_ok(C, {x, y, gamma, beta, mean, invstd}) && ((uintptr_t)y16 & 7) == 0)
        hipLaunchKernelGGL(bn_apply_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, x, M,
                           C, gamma, beta, mean, invstd, y, relu, y16);
    else
        hipLaunchKernelGGL(bn_apply_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, M, C,
                           gamma, beta, mean, invstd, y, relu, y16);
    return hipGetLastError();
}

hipError_t launch_bn_bwd(const float* x, const float* dy, const float* relu_y, long M, int C,
                         const float* gamma, const float* mean, const float* invstd, float* dx,
                         float* dgamma, float* dbeta, int accumulate, float* ws, hipStream_t s,
                         uint16_t* dx16) {
    const ColPlan p = col_plan(M, C, vec4_ok(C, {x, dy, relu_y, mean, invstd}) ? 4 : 1);
    float* p0 = ws;
    float* p1 = ws + (size_t)p.nb * C;
    launch_partial<MODE_BNBWD>(p, dy, x, relu_y, mean, invstd, M, C, p0, p1, s);
    launch_final<FIN_SUM2>(p, p0, p1, M, C, 0.f, dbeta, dgamma, s);
    if (!dx) return hipGetLastError();      // parameter gradients only
    size_t n = (size_t)M * C;
    if (vec4_ok(C, {x, dy, relu_y, dx, gamma, mean, invstd, dbeta, dgamma}) &&
        ((uintptr_t)dx16 & 7) == 0)
        hipLaunchKernelGGL(bn_bwd_apply_kernel<4>, dim3(ew_blocks(n / 4)), dim3(EW_THREADS), 0, s, x,
                           dy, relu_y, M, C, gamma, mean, invstd, dbeta, dgamma, dx, accumulate,
                           dx16);
    else
        hipLaunchKernelGGL(bn_bwd_apply_kernel<1>, dim3(ew_blocks(n)), dim3(EW_THREADS), 0, s, x, dy,
                           relu_y, M, C, gamma, mean, invstd, dbeta, dgamma, dx, accumulate, dx16);
    return hipGetLastError();
}

hipError_t launch_cast_bf16(const float* src, uint16_t* dst, size_t n, hipStream_t s) {
    const int vec = ((((uintptr_t)src) & 15) | (((uintptr_t)dst) & 7)) == 0;
    hipLaunchKernelGGL(cast_bf16_kernel, dim3(ew_blocks(vec ? (n + 3) / 4 : n)), dim3(EW_THREADS), 0,
                       s, src, dst, n, vec);
    return hipGetLastError();
}

hipError_t launch_pad_channels(const float* src, float* dst, uint16_t* dst16, size_t rows, int C,
                               int Cp, hipStream_t s) {
    hipLaunchKernelGGL(pad_channels_kernel, dim3(ew_blocks(rows * Cp)), dim3(EW_THREADS), 0, s, src,
                       dst, dst16, rows, C, Cp);
    return hipGetLastError();
}

hipError_t launch_unpad_channels(const float* src, float* dst, size_t rows, int C, int Cp,
                                 hipStream_t s) {
    hipLaunchKernelGGL(unpad_channels_kernel, dim3(ew_blocks(rows * C)), dim3(EW_THREADS), 0, s, src,
                       dst, rows, C, Cp);
    return hipGetLastError();
}

hipError_t launch_cast_bf16_t(const float* src, uint16_t* dst, const WtLayer* table,
                              int nlayers, int tiles, hipStream_t s) {
    if (nlayers <= 0 || tiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(cast_bf16_t_kernel, dim3(tiles), dim3(256), 0, s, src, dst, table,
                       nlayers);
    return hipGetLastError();
}

hipError_t launch_softmax_ce(const float* z, const int32_t* labels, int B, int K, float* loss,
                             float* dz, float* ws, hipStream_t s) {
    hipLaunchKernelGGL(softmax_ce_kernel, dim3(B), dim3(EW_THREADS), 0, s, z, labels, B, K, ws, dz);
    hipLaunchKernelGGL(mean_rows_kernel, dim3(1), dim3(64), 0, s, ws, B, loss);
    return hipGetLastError();
}

}  // namespace hp
