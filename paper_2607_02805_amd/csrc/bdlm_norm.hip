// bdlm_norm.hip -- gfx950 kernel for the gated RMS normalisation that follows the scan
// in a Mamba-2 mixer (App. C; the Mamba-2 output path): per token,
//   g = y * silu(z),  out = w * g / sqrt(mean over the channel group of g^2 + eps),
// over nheads * 64 channels in ngroups groups of whole heads.
//
// One workgroup per token (grid-stride over tokens).  Thread tid holds channel quads
// q = tid + 256 i in registers: 16 consecutive lanes cover one head (64 channels),
// so a 16-lane DPP reduction gives each head's sum of squares, which goes to LDS; after a
// barrier one thread per group adds its heads in order and stores the group's scale,
// and after a second barrier every thread scales its quads and stores them.  Every
// output element is written by the thread that read its y, so out may be y itself.
// All of a token's loads are issued before any of them is used (quads past the end
// read a zero chunk: no load sits under a branch), and the group sums read their
// heads eight at a time.  The sums are taken in a fixed order: the result does not
// depend on the launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_device.h"
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
    int32_t z_rows;                // 1: zs_b == len * zs_t, token tok's row at tok * zs_t
    float eps;
};

__device__ __forceinline__ float silu(float v) { return v / (1.f + expf(-v)); }

typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));
__device__ const v4f kZeroQuad = {0.f, 0.f, 0.f, 0.f};
typedef __attribute__((address_space(1))) const v4f g_f4;
typedef __attribute__((address_space(1))) const v2u g_u2;
__device__ __forceinline__ float4 f4(v4f v) { return float4{v.x, v.y, v.z, v.w}; }

// z quad at element offset off (bf16: 8 bytes, fp32: 16 bytes), or zeros when !ok
template <bool BF16>
__device__ __forceinline__ float4 load_z(const NormArgs &a, int64_t off, bool ok) {
    if constexpr (BF16) {
        const v2u u = *(ok ? (const g_u2 *)(static_cast<const uint16_t *>(a.z) + off)
                           : (const g_u2 *)(&kZeroQuad));
        return float4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                      __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
    } else {
        return f4(*(ok ? (const g_f4 *)(static_cast<const float *>(a.z) + off)
                       : (const g_f4 *)(&kZeroQuad)));
    }
}

template <int kQPT, bool BF16>
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
        float4 yv[kQPT], zv[kQPT];
#pragma unroll
        for (int i = 0; i < kQPT; ++i) {
            const int q = tid + kNT * i;
            const bool ok = q < a.nq;
            yv[i] = f4(*(ok ? (const g_f4 *)(yr + 4 * q) : (const g_f4 *)(&kZeroQuad)));
            zv[i] = load_z<BF16>(a, zr + 4 * q, ok);
        }
        float4 g[kQPT];
#pragma unroll
        for (int i = 0; i < kQPT; ++i) {
            const int q = tid + kNT * i;
            g[i] = float4{yv[i].x * silu(zv[i].x), yv[i].y * silu(zv[i].y),
                          yv[i].z * silu(zv[i].z), yv[i].w * silu(zv[i].w)};
            // one head = 16 consecutive lanes (q = tid + 256 i, nq a multiple of 16):
            // the reduction stays inside a head, and a head is all in or all out
            float s = g[i].x * g[i].x + g[i].y * g[i].y + g[i].z * g[i].z + g[i].w * g[i].w;
            s += dpp<0xb1, 0xf, false>(s);    // quad_perm [1,0,3,2]
            s += dpp<0x4e, 0xf, false>(s);    // quad_perm [2,3,0,1]: quad sums
            s += dpp<0x141, 0xf, false>(s);   // row_half_mirror: sums of 8
            s += dpp<0x140, 0xf, false>(s);   // row_mirror: sums of 16 in every lane
            if (q < a.nq && (tid & 15) == 0) sHead[q >> 4] = s;
        }
        __syncthreads();
        if (tid < a.ngroups) {
            // the group's heads in order, eight LDS reads in flight at a time
            const float *hs = sHead + tid * a.hpg;
            float ss = 0.f;
            int k = 0;
            for (; k + 8 <= a.hpg; k += 8) {
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = hs[k + e];
#pragma unroll
                for (int e = 0; e < 8; ++e) ss += v[e];
            }
            for (; k < a.hpg; ++k) ss += hs[k];
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

template <bool BF16>
hipError_t launch_norm(int per, const NormArgs &a, dim3 g, dim3 blk, hipStream_t s) {
    if (per <= 1) hipLaunchKernelGGL((bdlm_gated_rmsnorm_kernel<1, BF16>), g, blk, 0, s, a);
    else if (per <= 2) hipLaunchKernelGGL((bdlm_gated_rmsnorm_kernel<2, BF16>), g, blk, 0, s, a);
    else if (per <= 4) hipLaunchKernelGGL((bdlm_gated_rmsnorm_kernel<4, BF16>), g, blk, 0, s, a);
    else if (per <= 8) hipLaunchKernelGGL((bdlm_gated_rmsnorm_kernel<8, BF16>), g, blk, 0, s, a);
    else if (per <= 16) hipLaunchKernelGGL((bdlm_gated_rmsnorm_kernel<16, BF16>), g, blk, 0, s, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
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
    a.z_rows = n.zs_b == n.len * n.zs_t ? 1 : 0;
    a.eps = n.eps;
    const int64_t grid = a.ntok < (int64_t(1) << 20) ? a.ntok : (int64_t(1) << 20);
    const dim3 g(static_cast<unsigned>(grid)), blk(kNT);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int per = (a.nq + kNT - 1) / kNT;   // <= 16 (nheads <= 256)
    const hipError_t e = n.bf16 ? launch_norm<true>(per, a, g, blk, s) : launch_norm<false>(per, a, g, blk, s);
    if (e == hipErrorInvalidValue) return BDLM_E_SHAPE;
    return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

}  // namespace bdlm
