// WSP update kernels (gfx950): local update + wave accumulation, push, pull,
// and the three fused at a wave end.
//
// All three stream flat fp32 parameter vectors once, so they are HBM-bound:
// float4 accesses (four per thread on long vectors, all loads issued before the
// first use), one workgroup per 1024 (or 256) float4 of the vector, and a
// scalar tail for lengths that are not multiples of 4.
// Every vector is streamed once per kernel and not read again before other
// kernels have passed through the caches, so the loads are non-temporal.  The arithmetic
// is fixed to one IEEE fp32 operation at a time (contraction into fused
// multiply-add is switched off for this file), so the result is bit-identical to any
// other implementation that performs the same operations in the same order:
//   u = (-lr) * g;   new = newest + u;   u~ = u  or  u~ + u;   w_g = w_g + u~.
#include "kernels.h"

// One rounding per operation: never fuse a multiply and an add into an FMA here.
#pragma clang fp contract(off)

namespace hp {
namespace {

constexpr int WSP_THREADS = 256;
// float4 per thread per iteration: 4 for long vectors (all loads issued
// before the first use), 1 for short ones, where more workgroups start sooner.
constexpr size_t WSP_LONG = size_t(1) << 20;     // float4 elements (16 MB)

inline int wsp_unroll(size_t n4) { return n4 >= WSP_LONG ? 4 : 1; }

// One pass: every workgroup streams U * WSP_THREADS float4 once (the grid-stride
// loop below then runs one iteration).  Measured on the 143.7 M-parameter
// VGG-19 vectors, this keeps more DRAM requests in flight than a grid capped
// at 16 workgroups per CU looping over the vector (local update 72 -> 77 %,
// fused wave end 69 -> 74 % of 8 TB/s).
inline int wsp_blocks(size_t n4, int unroll) {
    size_t b = (n4 + (size_t)WSP_THREADS * unroll - 1) / ((size_t)WSP_THREADS * unroll);
    if (b > 0x7fffffff) b = 0x7fffffff;
    return (int)(b ? b : 1);
}

__device__ __forceinline__ float mul_rn(float a, float b) { return a * b; }
__device__ __forceinline__ float add_rn(float a, float b) { return a + b; }

typedef float fx4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ld4(const float4* p) {
    const fx4 v = __builtin_nontemporal_load(reinterpret_cast<const fx4*>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}
// non-temporal store: the copy's destination is not read again soon
__device__ __forceinline__ void st4_nt(float4* p, float4 v) {
    fx4 t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<fx4*>(p));
}

// Vector part: workgroup b's iteration covers U * blockDim.x consecutive
// float4 elements starting at (it * gridDim.x + b) * U * blockDim.x; thread t
// takes elements base + k * blockDim.x (k < U), so every load instruction of a
// wave reads 1 KB contiguous.
#define WSP_VECTOR_LOOP(n4)                                                               \
    const size_t stride = (size_t)gridDim.x * blockDim.x;                                 \
    for (size_t base = (size_t)blockIdx.x * blockDim.x * U + threadIdx.x; base < (n4);    \
         base += stride * U)

template <bool FIRST, int U>
__global__ void __launch_bounds__(WSP_THREADS)
local_update_kernel(const float* __restrict__ g, const float* newest, float* dst,
                    float* __restrict__ ut, size_t n, float neg_lr, int vec) {
    // newest and dst may alias (wave length 1): each element is read before it
    // is written by the same thread.
    const size_t n4 = vec ? n / 4 : 0;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const float4* w4 = reinterpret_cast<const float4*>(newest);
    float4* d4 = reinterpret_cast<float4*>(dst);
    float4* u4 = reinterpret_cast<float4*>(ut);
    WSP_VECTOR_LOOP(n4) {
        float4 gv[U], wv[U], av[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i < n4) {
                gv[k] = ld4(g4 + i);
                wv[k] = ld4(w4 + i);
                if (!FIRST) av[k] = ld4(u4 + i);
            }
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i >= n4) break;
            float4 u;
            u.x = mul_rn(neg_lr, gv[k].x); u.y = mul_rn(neg_lr, gv[k].y);
            u.z = mul_rn(neg_lr, gv[k].z); u.w = mul_rn(neg_lr, gv[k].w);
            float4 nw;
            nw.x = add_rn(wv[k].x, u.x); nw.y = add_rn(wv[k].y, u.y);
            nw.z = add_rn(wv[k].z, u.z); nw.w = add_rn(wv[k].w, u.w);
            d4[i] = nw;
            if (FIRST) {
                u4[i] = u;
            } else {
                float4 a = av[k];
                a.x = add_rn(a.x, u.x); a.y = add_rn(a.y, u.y);
                a.z = add_rn(a.z, u.z); a.w = add_rn(a.w, u.w);
                u4[i] = a;
            }
        }
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float u = mul_rn(neg_lr, g[i]);
        dst[i] = add_rn(newest[i], u);
        ut[i] = FIRST ? u : add_rn(ut[i], u);
    }
}

// Local update with momentum (heavy ball, no dampening): v = mu * v + g,
// u = (-lr) * v, then as above.  One rounding per operation.
template <bool FIRST, int U>
__global__ void __launch_bounds__(WSP_THREADS)
local_update_momentum_kernel(const float* __restrict__ g, const float* newest, float* dst,
                             float* __restrict__ ut, float* __restrict__ vel, size_t n,
                             float neg_lr, float mu, int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const float4* w4 = reinterpret_cast<const float4*>(newest);
    float4* d4 = reinterpret_cast<float4*>(dst);
    float4* u4 = reinterpret_cast<float4*>(ut);
    float4* v4 = reinterpret_cast<float4*>(vel);
    WSP_VECTOR_LOOP(n4) {
        float4 gv[U], wv[U], vv[U], av[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i < n4) {
                gv[k] = ld4(g4 + i);
                wv[k] = ld4(w4 + i);
                vv[k] = ld4(v4 + i);
                if (!FIRST) av[k] = ld4(u4 + i);
            }
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i >= n4) break;
            float4 v;
            v.x = add_rn(mul_rn(mu, vv[k].x), gv[k].x); v.y = add_rn(mul_rn(mu, vv[k].y), gv[k].y);
            v.z = add_rn(mul_rn(mu, vv[k].z), gv[k].z); v.w = add_rn(mul_rn(mu, vv[k].w), gv[k].w);
            v4[i] = v;
            float4 u;
            u.x = mul_rn(neg_lr, v.x); u.y = mul_rn(neg_lr, v.y);
            u.z = mul_rn(neg_lr, v.z); u.w = mul_rn(neg_lr, v.w);
            float4 nw;
            nw.x = add_rn(wv[k].x, u.x); nw.y = add_rn(wv[k].y, u.y);
            nw.z = add_rn(wv[k].z, u.z); nw.w = add_rn(wv[k].w, u.w);
            d4[i] = nw;
            if (FIRST) {
                u4[i] = u;
            } else {
                float4 a = av[k];
                a.x = add_rn(a.x, u.x); a.y = add_rn(a.y, u.y);
                a.z = add_rn(a.z, u.z); a.w = add_rn(a.w, u.w);
                u4[i] = a;
            }
        }
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const float v = add_rn(mul_rn(mu, vel[i]), g[i]);
        vel[i] = v;
        const float u = mul_rn(neg_lr, v);
        dst[i] = add_rn(newest[i], u);
        ut[i] = FIRST ? u : add_rn(ut[i], u);
    }
}

template <int U>
__global__ void __launch_bounds__(WSP_THREADS)
push_kernel(float* __restrict__ wg, const float* __restrict__ ut, size_t n, int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    float4* w4 = reinterpret_cast<float4*>(wg);
    const float4* u4 = reinterpret_cast<const float4*>(ut);
    WSP_VECTOR_LOOP(n4) {
        float4 a[U], b[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i < n4) { a[k] = ld4(w4 + i); b[k] = ld4(u4 + i); }
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i >= n4) break;
            float4 v = a[k];
            v.x = add_rn(v.x, b[k].x); v.y = add_rn(v.y, b[k].y);
            v.z = add_rn(v.z, b[k].z); v.w = add_rn(v.w, b[k].w);
            w4[i] = v;
        }
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        wg[i] = add_rn(wg[i], ut[i]);
}

template <int U>
__global__ void __launch_bounds__(WSP_THREADS)
copy_kernel(const float* __restrict__ src, float* __restrict__ dst, size_t n, int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    const float4* s4 = reinterpret_cast<const float4*>(src);
    float4* d4 = reinterpret_cast<float4*>(dst);
    WSP_VECTOR_LOOP(n4) {
        float4 a[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i < n4) a[k] = ld4(s4 + i);
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i < n4) st4_nt(d4 + i, a[k]);
        }
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
}

// Wave end in one pass: the local update of the minibatch that completes a
// wave, the push of the wave's aggregate and, when the clock-bound gate opens
// at once, the pull.  Per element, in this order (the order of the three
// separate kernels above, so the results are bit-identical to them):
//   (momentum) v = mu * v + g;   u = (-lr) * (g or v);
//   u~ = u or u~ + u;   w_g = w_g + u~;
//   slot = w_g (PULL)  or  newest + u.
// With PULL the newest ring version is not read: the pull replaces the
// slot's new version by w_g.  Bytes per parameter: read g, u~ (unless FIRST),
// w_g, newest (unless PULL), v (MOM); write u~, w_g, the slot, v (MOM).
template <bool FIRST, bool PULL, bool MOM, int U>
__global__ void __launch_bounds__(WSP_THREADS)
wave_end_kernel(const float* __restrict__ g, const float* newest, float* dst,
                float* __restrict__ ut, float* __restrict__ vel, float* __restrict__ wg,
                size_t n, float neg_lr, float mu, int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const float4* w4 = reinterpret_cast<const float4*>(newest);
    float4* d4 = reinterpret_cast<float4*>(dst);
    float4* u4 = reinterpret_cast<float4*>(ut);
    float4* v4 = reinterpret_cast<float4*>(vel);
    float4* s4 = reinterpret_cast<float4*>(wg);
    WSP_VECTOR_LOOP(n4) {
        float4 gv[U], wv[U], av[U], vv[U], sv[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i < n4) {
                gv[k] = ld4(g4 + i);
                if (!PULL) wv[k] = ld4(w4 + i);
                if (!FIRST) av[k] = ld4(u4 + i);
                if (MOM) vv[k] = ld4(v4 + i);
                sv[k] = ld4(s4 + i);
            }
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const size_t i = base + (size_t)k * blockDim.x;
            if (i >= n4) break;
            float4 d = gv[k];
            if (MOM) {
                d.x = add_rn(mul_rn(mu, vv[k].x), gv[k].x);
                d.y = add_rn(mul_rn(mu, vv[k].y), gv[k].y);
                d.z = add_rn(mul_rn(mu, vv[k].z), gv[k].z);
                d.w = add_rn(mul_rn(mu, vv[k].w), gv[k].w);
                v4[i] = d;
            }
            float4 u;
            u.x = mul_rn(neg_lr, d.x); u.y = mul_rn(neg_lr, d.y);
            u.z = mul_rn(neg_lr, d.z); u.w = mul_rn(neg_lr, d.w);
            if (!PULL) {
                float4 nw;
                nw.x = add_rn(wv[k].x, u.x); nw.y = add_rn(wv[k].y, u.y);
                nw.z = add_rn(wv[k].z, u.z); nw.w = add_rn(wv[k].w, u.w);
                d4[i] = nw;
            }
            float4 a = u;
            if (!FIRST) {
                a.x = add_rn(av[k].x, u.x); a.y = add_rn(av[k].y, u.y);
                a.z = add_rn(av[k].z, u.z); a.w = add_rn(av[k].w, u.w);
            }
            u4[i] = a;
            float4 w = sv[k];
            w.x = add_rn(w.x, a.x); w.y = add_rn(w.y, a.y);
            w.z = add_rn(w.z, a.z); w.w = add_rn(w.w, a.w);
            s4[i] = w;
            if (PULL) d4[i] = w;
        }
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float d = g[i];
        if (MOM) {
            d = add_rn(mul_rn(mu, vel[i]), g[i]);
            vel[i] = d;
        }
        const float u = mul_rn(neg_lr, d);
        if (!PULL) dst[i] = add_rn(newest[i], u);
        const float a = FIRST ? u : add_rn(ut[i], u);
        ut[i] = a;
        const float w = add_rn(wg[i], a);
        wg[i] = w;
        if (PULL) dst[i] = w;
    }
}

template <bool FIRST, bool PULL, bool MOM>
void launch_wave_end_t(dim3 grid, dim3 block, int u, hipStream_t s, const float* g,
                       const float* newest, float* dst, float* ut, float* vel, float* wg,
                       size_t n, float neg_lr, float mu, int vec) {
    if (u == 4)
        hipLaunchKernelGGL((wave_end_kernel<FIRST, PULL, MOM, 4>), grid, block, 0, s, g, newest,
                           dst, ut, vel, wg, n, neg_lr, mu, vec);
    else
        hipLaunchKernelGGL((wave_end_kernel<FIRST, PULL, MOM, 1>), grid, block, 0, s, g, newest,
                           dst, ut, vel, wg, n, neg_lr, mu, vec);
}

inline int aligned16(const void* a, const void* b, const void* c = nullptr,
                     const void* d = nullptr) {
    uintptr_t u = (uintptr_t)a | (uintptr_t)b | (uintptr_t)c | (uintptr_t)d;
    return (u & 15) == 0;
}

}  // namespace

hipError_t launch_wsp_local_update(const float* g, const float* newest, float* dst, float* ut,
                                   size_t n, float lr, int first, hipStream_t s) {
    const float neg_lr = -lr;
    const int vec = aligned16(g, newest, dst, ut);
    const size_t n4 = vec ? n / 4 : n;
    const int u = wsp_unroll(n4);
    const dim3 grid(wsp_blocks(n4, u)), block(WSP_THREADS);
    if (first && u == 4)
        hipLaunchKernelGGL((local_update_kernel<true, 4>), grid, block, 0, s, g, newest, dst, ut, n,
                           neg_lr, vec);
    else if (first)
        hipLaunchKernelGGL((local_update_kernel<true, 1>), grid, block, 0, s, g, newest, dst, ut, n,
                           neg_lr, vec);
    else if (u == 4)
        hipLaunchKernelGGL((local_update_kernel<false, 4>), grid, block, 0, s, g, newest, dst, ut, n,
                           neg_lr, vec);
    else
        hipLaunchKernelGGL((local_update_kernel<false, 1>), grid, block, 0, s, g, newest, dst, ut, n,
                           neg_lr, vec);
    return hipGetLastError();
}

hipError_t launch_wsp_local_update_momentum(const float* g, const float* newest, float* dst,
                                            float* ut, float* vel, size_t n, float lr, float mu,
                                            int first, hipStream_t s) {
    const float neg_lr = -lr;
    const int vec = aligned16(g, newest, dst, ut) && aligned16(vel, vel);
    const size_t n4 = vec ? n / 4 : n;
    const int u = wsp_unroll(n4);
    const dim3 grid(wsp_blocks(n4, u)), block(WSP_THREADS);
    if (first && u == 4)
        hipLaunchKernelGGL((local_update_momentum_kernel<true, 4>), grid, block, 0, s, g, newest,
                           dst, ut, vel, n, neg_lr, mu, vec);
    else if (first)
        hipLaunchKernelGGL((local_update_momentum_kernel<true, 1>), grid, block, 0, s, g, newest,
                           dst, ut, vel, n, neg_lr, mu, vec);
    else if (u == 4)
        hipLaunchKernelGGL((local_update_momentum_kernel<false, 4>), grid, block, 0, s, g, newest,
                           dst, ut, vel, n, neg_lr, mu, vec);
    else
        hipLaunchKernelGGL((local_update_momentum_kernel<false, 1>), grid, block, 0, s, g, newest,
                           dst, ut, vel, n, neg_lr, mu, vec);
    return hipGetLastError();
}

hipError_t launch_wsp_push(float* wg, const float* ut, size_t n, hipStream_t s) {
    const int vec = aligned16(wg, ut);
    const size_t n4 = vec ? n / 4 : n;
    const int u = wsp_unroll(n4);
    const dim3 grid(wsp_blocks(n4, u)), block(WSP_THREADS);
    if (u == 4)
        hipLaunchKernelGGL(push_kernel<4>, grid, block, 0, s, wg, ut, n, vec);
    else
        hipLaunchKernelGGL(push_kernel<1>, grid, block, 0, s, wg, ut, n, vec);
    return hipGetLastError();
}

hipError_t launch_wsp_copy(const float* src, float* dst, size_t n, hipStream_t s) {
    const int vec = aligned16(src, dst);
    const size_t n4 = vec ? n / 4 : n;
    const int u = wsp_unroll(n4);
    const dim3 grid(wsp_blocks(n4, u)), block(WSP_THREADS);
    if (u == 4)
        hipLaunchKernelGGL(copy_kernel<4>, grid, block, 0, s, src, dst, n, vec);
    else
        hipLaunchKernelGGL(copy_kernel<1>, grid, block, 0, s, src, dst, n, vec);
    return hipGetLastError();
}

hipError_t launch_wsp_wave_end(const float* g, const float* newest, float* dst, float* ut,
                               float* vel, float* wg, size_t n, float lr, float mu, int first,
                               int pull, hipStream_t s) {
    const float neg_lr = -lr;
    const bool mom = vel != nullptr;
    const int vec = aligned16(g, newest, dst, ut) && aligned16(wg, mom ? vel : wg);
    const size_t n4 = vec ? n / 4 : n;
    const int u = wsp_unroll(n4);
    const dim3 grid(wsp_blocks(n4, u)), block(WSP_THREADS);
    const int sel = (first ? 4 : 0) | (pull ? 2 : 0) | (mom ? 1 : 0);
#define HP_WAVE_END(F, P, M) \
    launch_wave_end_t<F, P, M>(grid, block, u, s, g, newest, dst, ut, vel, wg, n, neg_lr, mu, vec)
    switch (sel) {
        case 0: HP_WAVE_END(false, false, false); break;
        case 1: HP_WAVE_END(false, false, true); break;
        case 2: HP_WAVE_END(false, true, false); break;
        case 3: HP_WAVE_END(false, true, true); break;
        case 4: HP_WAVE_END(true, false, false); break;
        case 5: HP_WAVE_END(true, false, true); break;
        case 6: HP_WAVE_END(true, true, false); break;
        default: HP_WAVE_END(true, true, true); break;
    }
#undef HP_WAVE_END
    return hipGetLastError();
}

}  // namespace hp
