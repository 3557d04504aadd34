// WSP update kernels (gfx950): local update + wave accumulation, push, pull.
//
// All three stream flat fp32 parameter vectors once, so they are HBM-bound:
// float4 accesses, a grid of a few workgroups per CU striding over the vector,
// and a scalar tail for lengths that are not multiples of 4.  The arithmetic
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

inline int wsp_blocks(size_t n4) {
    size_t b = (n4 + WSP_THREADS - 1) / WSP_THREADS;
    if (b > 4096) b = 4096;      // 16 workgroups per CU, grid-stride beyond that
    return (int)(b ? b : 1);
}

__device__ __forceinline__ float mul_rn(float a, float b) { return a * b; }
__device__ __forceinline__ float add_rn(float a, float b) { return a + b; }

template <bool FIRST>
__global__ void local_update_kernel(const float* __restrict__ g, const float* newest,
                                    float* dst, float* __restrict__ ut, size_t n, float neg_lr,
                                    int vec) {
    // newest and dst may alias (wave length 1): each element is read before it
    // is written by the same thread.
    const size_t n4 = vec ? n / 4 : 0;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const float4* g4 = reinterpret_cast<const float4*>(g);
    const float4* w4 = reinterpret_cast<const float4*>(newest);
    float4* d4 = reinterpret_cast<float4*>(dst);
    float4* u4 = reinterpret_cast<float4*>(ut);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 gv = g4[i];
        float4 wv = w4[i];
        float4 u;
        u.x = mul_rn(neg_lr, gv.x); u.y = mul_rn(neg_lr, gv.y);
        u.z = mul_rn(neg_lr, gv.z); u.w = mul_rn(neg_lr, gv.w);
        float4 nw;
        nw.x = add_rn(wv.x, u.x); nw.y = add_rn(wv.y, u.y);
        nw.z = add_rn(wv.z, u.z); nw.w = add_rn(wv.w, u.w);
        d4[i] = nw;
        if (FIRST) {
            u4[i] = u;
        } else {
            float4 a = u4[i];
            a.x = add_rn(a.x, u.x); a.y = add_rn(a.y, u.y);
            a.z = add_rn(a.z, u.z); a.w = add_rn(a.w, u.w);
            u4[i] = a;
        }
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float u = mul_rn(neg_lr, g[i]);
        dst[i] = add_rn(newest[i], u);
        ut[i] = FIRST ? u : add_rn(ut[i], u);
    }
}

__global__ void push_kernel(float* __restrict__ wg, const float* __restrict__ ut, size_t n,
                            int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    float4* w4 = reinterpret_cast<float4*>(wg);
    const float4* u4 = reinterpret_cast<const float4*>(ut);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 a = w4[i], b = u4[i];
        a.x = add_rn(a.x, b.x); a.y = add_rn(a.y, b.y);
        a.z = add_rn(a.z, b.z); a.w = add_rn(a.w, b.w);
        w4[i] = a;
    }
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        wg[i] = add_rn(wg[i], ut[i]);
}

__global__ void copy_kernel(const float* __restrict__ src, float* __restrict__ dst, size_t n,
                            int vec) {
    const size_t n4 = vec ? n / 4 : 0;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    const float4* s4 = reinterpret_cast<const float4*>(src);
    float4* d4 = reinterpret_cast<float4*>(dst);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) d4[i] = s4[i];
    for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
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
    const int blocks = wsp_blocks(vec ? n / 4 : n);
    if (first)
        hipLaunchKernelGGL(local_update_kernel<true>, dim3(blocks), dim3(WSP_THREADS), 0, s, g,
                           newest, dst, ut, n, neg_lr, vec);
    else
        hipLaunchKernelGGL(local_update_kernel<false>, dim3(blocks), dim3(WSP_THREADS), 0, s, g,
                           newest, dst, ut, n, neg_lr, vec);
    return hipGetLastError();
}

hipError_t launch_wsp_push(float* wg, const float* ut, size_t n, hipStream_t s) {
    const int vec = aligned16(wg, ut);
    hipLaunchKernelGGL(push_kernel, dim3(wsp_blocks(vec ? n / 4 : n)), dim3(WSP_THREADS), 0, s, wg,
                       ut, n, vec);
    return hipGetLastError();
}

hipError_t launch_wsp_copy(const float* src, float* dst, size_t n, hipStream_t s) {
    const int vec = aligned16(src, dst);
    hipLaunchKernelGGL(copy_kernel, dim3(wsp_blocks(vec ? n / 4 : n)), dim3(WSP_THREADS), 0, s, src,
                       dst, n, vec);
    return hipGetLastError();
}

}  // namespace hp
