// bdlm_norm.hip -- gfx950 kernel for the gated RMS normalisation that follows the scan
// in a Mamba-2 mixer (App. C; the Mamba-2 output path): per token,
//   g = y * silu(z),  out = w * g / sqrt(mean over the channel group of g^2 + eps),
// over nheads * 64 channels in ngroups groups of whole heads.
//
// One workgroup per token (grid-stride over tokens).  Thread tid holds channel quads
// q = tid + 256 i in registers: 16 consecutive lanes cover one head (64 channels),
// so a 16-lane butterfly gives each head's sum of squares, which goes to LDS; after a
// barrier one thread per group adds its heads in order and stores the group's scale,
// and after a second barrier every thread scales its quads and stores them.  Every
// output element is written by the thread that read its y, so out may be y itself.
// The sums are taken in a fixed order: the result does not depend on the launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

constexpr int kNT = 256;           // threads per workgroup (one token at a time)
// quads per thread (QPT, a template argument): 1, 2, 4, 8 or 16 -- up to 16384 channels

struct NormArgs {
    const float *y;
    const void *z;
    const float *w;
    float *out;
    int64_t zs_b, zs_t;            // z strides (elements)
    int64_t ntok, len;
    int32_t nq, gq;                // quads per token / per group
    int32_t ngroups, hpg;          // groups, heads per group
    int32_t bf16;
    int32_t z_rows;                // 1: zs_b == len * zs_t, token tok's row at tok * zs_t
    float eps;
};

__device__ __forceinline__ float silu(float v) { return v / (1.f + expf(-v)); }

__device__ __forceinline__ float4 load_z(const NormArgs &a, int64_t off) {
    if (a.bf16) {
        const uint2 u = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(a.z) + off);
        return float4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                      __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
    }
    return *reinterpret_cast<const float4 *>(static_cast<const float *>(a.z) + off);
}

template <int kQPT>
__global__ void __launch_bounds__(kNT) bdlm_gated_rmsnorm_kernel(const NormArgs a) {
    __shared__ float sHead[256];
    __shared__ float sScale[256];
    const int tid = threadIdx.x;
    const float inv_gs = 1.f / static_cast<float>(4 * a.gq);
    // per quad: its weights and its group (the same for every token)
    float4 wv[kQPT];
    int grp[kQPT];
#pragma unroll
    for (int i = 0; i < kQPT; ++i) {
        const int q = tid + kNT * i;
        wv[i] = q < a.nq ? *reinterpret_cast<const float4 *>(a.w + 4 * q) : float4{0.f, 0.f, 0.f, 0.f};
        grp[i] = q < a.nq ? q / a.gq : 0;
    }
    for (int64_t tok = blockIdx.x; tok < a.ntok; tok += gridDim.x) {
        const int64_t zr = a.z_rows ? tok * a.zs_t : (tok / a.len) * a.zs_b + (tok % a.len) * a.zs_t;
        const float *yr = a.y + tok * (4 * static_cast<int64_t>(a.nq));
        float4 g[kQPT];
#pragma unroll
        for (int i = 0; i < kQPT; ++i) {
            const int q = tid + kNT * i;
            g[i] = float4{0.f, 0.f, 0.f, 0.f};
            if (q < a.nq) {
                const float4 yv = *reinterpret_cast<const float4 *>(yr + 4 * q);
                const float4 zv = load_z(a, zr + 4 * q);
                g[i] = float4{yv.x * silu(zv.x), yv.y * silu(zv.y), yv.z * silu(zv.z),
                              yv.w * silu(zv.w)};
            }
            // one head = 16 consecutive lanes (q = tid + 256 i, nq a multiple of 16):
            // the butterfly stays inside a head, and a head is all in or all out
            float s = g[i].x * g[i].x + g[i].y * g[i].y + g[i].z * g[i].z + g[i].w * g[i].w;
            s += __shfl_xor(s, 1, 16);
            s += __shfl_xor(s, 2, 16);
            s += __shfl_xor(s, 4, 16);
            s += __shfl_xor(s, 8, 16);
            if (q < a.nq && (tid & 15) == 0) sHead[q >> 4] = s;
        }
        __syncthreads();
        if (tid < a.ngroups) {
            float ss = 0.f;
            for (int k = tid * a.hpg; k < (tid + 1) * a.hpg; ++k) ss += sHead[k];
            sScale[tid] = 1.f / sqrtf(ss * inv_gs + a.eps);
        }
        __syncthreads();
        float *orow = a.out + tok * (4 * static_cast<int64_t>(a.nq));
#pragma unroll
        for (int i = 0; i < kQPT; ++i) {
            const int q = tid + kNT * i;
            if (q < a.nq) {
                const float r = sScale[grp[i]];
                *reinterpret_cast<float4 *>(orow + 4 * q) = float4{
                    g[i].x * wv[i].x * r, g[i].y * wv[i].y * r, g[i].z * wv[i].z * r, g[i].w * wv[i].w * r};
            }
        }
        __syncthreads();   // sHead / sScale are rewritten for the next token
    }
}

}  // namespace

int launch_gated_rmsnorm(const NormLaunch &n, void *stream) {
    if (n.batch == 0 || n.len == 0) return BDLM_OK;
    NormArgs a;
    a.y = n.y;
    a.z = n.z;
    a.w = n.w;
    a.out = n.out;
    a.zs_b = n.zs_b;
    a.zs_t = n.zs_t;
    a.ntok = n.batch * n.len;
    a.len = n.len;
    a.nq = static_cast<int32_t>(n.nheads * 16);
    a.gq = static_cast<int32_t>(n.nheads / n.ngroups * 16);
    a.ngroups = static_cast<int32_t>(n.ngroups);
    a.hpg = static_cast<int32_t>(n.nheads / n.ngroups);
    a.bf16 = n.bf16;
    a.z_rows = n.zs_b == n.len * n.zs_t ? 1 : 0;
    a.eps = n.eps;
    const int64_t grid = a.ntok < (int64_t(1) << 20) ? a.ntok : (int64_t(1) << 20);
    const dim3 g(static_cast<unsigned>(grid)), blk(kNT);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int per = (a.nq + kNT - 1) / kNT;   // <= 16 (nheads <= 256)
    if (per <= 1) hipLaunchKernelGGL(bdlm_gated_rmsnorm_kernel<1>, g, blk, 0, s, a);
    else if (per <= 2) hipLaunchKernelGGL(bdlm_gated_rmsnorm_kernel<2>, g, blk, 0, s, a);
    else if (per <= 4) hipLaunchKernelGGL(bdlm_gated_rmsnorm_kernel<4>, g, blk, 0, s, a);
    else if (per <= 8) hipLaunchKernelGGL(bdlm_gated_rmsnorm_kernel<8>, g, blk, 0, s, a);
    else if (per <= 16) hipLaunchKernelGGL(bdlm_gated_rmsnorm_kernel<16>, g, blk, 0, s, a);
    else return BDLM_E_SHAPE;
    return hipGetLastError() == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

}  // namespace bdlm
