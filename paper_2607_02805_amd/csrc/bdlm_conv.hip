// bdlm_conv.hip -- the convolution part of the Mamba boundary state on gfx950: a
// width-4 depthwise causal convolution with SiLU over the x, B and C channels of the
// active block (the Mamba-2 mixer's convolution, App. C), in two versions -- the
// forward branch continues from the cached last three input rows, the reverse branch
// (local to the block, Sec. 4) is zero-padded past the block's end -- and, for a
// commit, the cache rows replaced by the last three rows of (cache ++ block).
//
// One thread per (batch row, four channels, 2-token tile); channels are contiguous
// across threads, so a token's row is one coalesced read of 8 (bf16) or 16 (fp32) bytes
// per thread.  A thread loads its tile with a three-row halo on each side (cached rows
// before the block, zeros after it) and computes both branches from registers; a
// commit's new cache rows are written by a second small kernel once every tile has
// read the old ones.  Every row is read as the sum of two unconditional loads, the
// cached row and the input row, each replaced by a zero chunk where it does not apply,
// so all loads of a thread are in flight at once.  Outputs are fp32 in the scan's
// input layouts (plus dt widened to fp32), consumed by the block kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

struct ConvArgs {
    const void *x, *Bm, *Cm, *dt;
    int64_t xs_b, xs_t, xs_h, dts_b, dts_t, bcs_b, bcs_t, bcs_g;
    const float *w, *bias;      // [channels][4] (w[c][3] on the current token), [channels]
    float *cache;               // [nslots][3][channels], row 0 the oldest input
    float *out;                 // fp32: xf, bf, cf, xr, br, cr, dtf (see conv_workspace)
    int32_t batch, L, nheads, ngroups, dstate, bf16, commit, use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

__device__ __forceinline__ float load_act(const void *p, int64_t i, int bf16) {
    if (bf16)
        return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t *>(p)[i]) << 16);
    return static_cast<const float *>(p)[i];
}

typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));
__device__ const v4f kZero4 = {0.f, 0.f, 0.f, 0.f};
typedef __attribute__((address_space(1))) const v4f g_v4f;
typedef __attribute__((address_space(1))) const v2u g_v2u;
typedef __attribute__((address_space(1))) const uint16_t g_u16;
typedef __attribute__((address_space(1))) const float g_f32;

// One activation (element i of p) as a float, or zero when !ok (read from a zero chunk).
template <bool BF16>
__device__ __forceinline__ float load_act_or_zero(const void *p, int64_t i, bool ok) {
    if constexpr (BF16)
        return __uint_as_float(static_cast<uint32_t>(*(ok ? (const g_u16 *)(static_cast<const uint16_t *>(p) + i)
                                                          : (const g_u16 *)(&kZero4)))
                               << 16);
    else
        return *(ok ? (const g_f32 *)(static_cast<const float *>(p) + i) : (const g_f32 *)(&kZero4));
}
__device__ __forceinline__ float silu(float v) { return v / (1.f + expf(-v)); }

constexpr int kTT = 2;    // tokens per thread
constexpr int kCV = 4;    // channels per thread (never straddles x / B / C: their
                          // boundaries are multiples of 16 channels)
constexpr int kCT = 256;  // threads per workgroup

// Four consecutive activations of one token row (element i of p) as floats, or zeros
// when !ok (the load then reads a zero chunk).
template <bool BF16>
__device__ __forceinline__ v4f load_act4(const void *p, int64_t i, bool ok) {
    if constexpr (BF16) {
        const v2u u = *(ok ? (const g_v2u *)(static_cast<const uint16_t *>(p) + i)
                           : (const g_v2u *)(&kZero4));
        return v4f{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                   __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
    } else {
        return *(ok ? (const g_v4f *)(static_cast<const float *>(p) + i) : (const g_v4f *)(&kZero4));
    }
}

// grid: (channel blocks of kCT * kCV, batch rows, token tiles of kTT)
template <bool BF16>
__global__ void __launch_bounds__(kCT) bdlm_conv_kernel(const ConvArgs a) {
    const int HP = a.nheads * 64, GN = a.ngroups * a.dstate, CH = HP + 2 * GN;
    const int c = (blockIdx.x * kCT + threadIdx.x) * kCV;   // first of this thread's channels
    const int b = blockIdx.y;
    const int t0 = blockIdx.z * kTT;
    const int64_t L = a.L;
    const int64_t BL = static_cast<int64_t>(a.batch) * L;

    if (c >= CH) return;

    // where these channels live: input element offset of token 0, token stride, and
    // the fp32 output plane / offset of token 0 / token stride within the plane
    const void *src;
    int64_t in0, in_t;
    int plane;            // 0 x, 1 B, 2 C
    int64_t o0, o_t;
    if (c < HP) {
        src = a.x;
        in0 = b * a.xs_b + (c / 64) * a.xs_h + c % 64;
        in_t = a.xs_t;
        plane = 0;
        o0 = b * L * HP + c;
        o_t = HP;
    } else {
        const int j = (c - HP) % GN;
        plane = c < HP + GN ? 1 : 2;
        src = plane == 1 ? a.Bm : a.Cm;
        in0 = b * a.bcs_b + (j / a.dstate) * a.bcs_g + j % a.dstate;
        in_t = a.bcs_t;
        o0 = b * L * GN + j;
        o_t = GN;
    }
    // output planes: [xf | bf | cf | xr | br | cr | dtf]
    float *planes[6];
    planes[0] = a.out;
    planes[1] = planes[0] + BL * HP;
    planes[2] = planes[1] + BL * GN;
    planes[3] = planes[2] + BL * GN;
    planes[4] = planes[3] + BL * HP;
    planes[5] = planes[4] + BL * GN;
    float *of = planes[plane] + o0, *orv = planes[3 + plane] + o0;

    float w[kCV][4], bc[kCV];
#pragma unroll
    for (int e = 0; e < kCV; ++e) {
        const float4 wv = *reinterpret_cast<const float4 *>(a.w + static_cast<int64_t>(c + e) * 4);
        w[e][0] = wv.x;
        w[e][1] = wv.y;
        w[e][2] = wv.z;
        w[e][3] = wv.w;
        bc[e] = a.bias[c + e];
    }
    const int64_t slot = a.use_slots ? a.slots[b] : b;
    const float *crow = a.cache + slot * 3 * CH + c;

    // inputs u[t0 - 3 .. t0 + kTT + 2]: cached rows before token 0, zeros past L; each
    // row the sum of the cached-row load and the input-row load, one of them zeros
    v4f u[kTT + 6];
#pragma unroll
    for (int i = 0; i < kTT + 6; ++i) {
        const int64_t t = t0 - 3 + i;
        const int64_t tc = t < 0 ? 0 : (t < L ? t : L - 1);   // addresses stay in range
        const v4f cv = *(t < 0 ? (const g_v4f *)(crow + (t < 0 ? t + 3 : 0) * CH)
                               : (const g_v4f *)(&kZero4));
        u[i] = cv + load_act4<BF16>(src, in0 + tc * in_t, t >= 0 && t < L);
    }
    // dt widened to fp32 (heads c .. c + 3; nheads < CH): loaded with the rows, stored
    // at the end
    float dtw[kCV][kTT];
#pragma unroll
    for (int e = 0; e < kCV; ++e)
#pragma unroll
        for (int i = 0; i < kTT; ++i) {
            const bool ok = c + e < a.nheads && t0 + i < L;
            dtw[e][i] = load_act_or_zero<BF16>(a.dt, ok ? b * a.dts_b + (t0 + i) * a.dts_t + c + e : 0, ok);
        }
#pragma unroll
    for (int i = 0; i < kTT; ++i) {
        const int64_t t = t0 + i;
        if (t < L) {
            // forward: u[t-3 .. t]; reverse: u[t .. t+3] (zeros past the block's end)
            float vf[kCV], vr[kCV];
#pragma unroll
            for (int e = 0; e < kCV; ++e) {
                vf[e] = silu(bc[e] + w[e][0] * u[i][e] + w[e][1] * u[i + 1][e] +
                             w[e][2] * u[i + 2][e] + w[e][3] * u[i + 3][e]);
                vr[e] = silu(bc[e] + w[e][0] * u[i + 6][e] + w[e][1] * u[i + 5][e] +
                             w[e][2] * u[i + 4][e] + w[e][3] * u[i + 3][e]);
            }
            *reinterpret_cast<float4 *>(of + t * o_t) = float4{vf[0], vf[1], vf[2], vf[3]};
            *reinterpret_cast<float4 *>(orv + t * o_t) = float4{vr[0], vr[1], vr[2], vr[3]};
        }
    }
#pragma unroll
    for (int e = 0; e < kCV; ++e)
#pragma unroll
        for (int i = 0; i < kTT; ++i)
            if (c + e < a.nheads && t0 + i < L)
                a.out[2 * BL * CH + (b * L + t0 + i) * a.nheads + c + e] = dtw[e][i];
}

// A commit's cache rows: the last three rows of (cache ++ block), one thread per
// (batch row, channel).  A kernel of its own, launched after the convolution, so that
// no tile of the convolution can read rows it already replaced.
__global__ void __launch_bounds__(256) bdlm_conv_keep_kernel(const ConvArgs a) {
    const int HP = a.nheads * 64, GN = a.ngroups * a.dstate, CH = HP + 2 * GN;
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int b = blockIdx.y;
    if (c >= CH) return;
    const void *src;
    int64_t in0, in_t;
    if (c < HP) {
        src = a.x;
        in0 = b * a.xs_b + (c / 64) * a.xs_h + c % 64;
        in_t = a.xs_t;
    } else {
        const int j = (c - HP) % GN;
        src = c < HP + GN ? a.Bm : a.Cm;
        in0 = b * a.bcs_b + (j / a.dstate) * a.bcs_g + j % a.dstate;
        in_t = a.bcs_t;
    }
    const int64_t slot = a.use_slots ? a.slots[b] : b;
    float *crow = a.cache + slot * 3 * CH + c;
    float r[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int64_t t = static_cast<int64_t>(a.L) - 3 + k;   // < 0: an older cached row
        r[k] = t < 0 ? crow[(t + 3) * CH] : load_act(src, in0 + t * in_t, a.bf16);
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) crow[k * CH] = r[k];
}

}  // namespace

int launch_conv_block(const LaunchArgs &a, const float *w, const float *bias, float *conv_pool,
                      bool commit, void *ws, void *stream) {
    if (a.batch == 0 || a.L == 0) return BDLM_OK;
    ConvArgs k;
    k.x = a.x;
    k.Bm = a.Bm;
    k.Cm = a.Cm;
    k.dt = a.dt;
    k.xs_b = a.xs_b;
    k.xs_t = a.xs_t;
    k.xs_h = a.xs_h;
    k.dts_b = a.dts_b;
    k.dts_t = a.dts_t;
    k.bcs_b = a.bcs_b;
    k.bcs_t = a.bcs_t;
    k.bcs_g = a.bcs_g;
    k.w = w;
    k.bias = bias;
    k.cache = conv_pool;
    k.out = static_cast<float *>(ws);
    k.batch = a.batch;
    k.L = a.L;
    k.nheads = a.nheads;
    k.ngroups = a.ngroups;
    k.dstate = a.dstate;
    k.bf16 = a.bf16;
    k.commit = commit ? 1 : 0;
    k.use_slots = a.slots ? 1 : 0;
    for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i)
        k.slots[i] = (a.slots && i < a.batch) ? a.slots[i] : 0;
    const int ch = a.nheads * 64 + 2 * a.ngroups * a.dstate;
    if (a.bf16 && a.L <= 32) {
        // bf16 blocks of at most 32 tokens: the block kernels convolve while staging (no
        // workspace); a commit's cache rows are replaced once both launches have read them
        const int rc = launch_conv_fused(a, w, bias, conv_pool, commit, a.y != nullptr, stream);
        if (rc != BDLM_OK || !commit) return rc;
        hipLaunchKernelGGL(bdlm_conv_keep_kernel, dim3((ch + 255) / 256, a.batch), dim3(256), 0,
                           static_cast<hipStream_t>(stream), k);
        return hipGetLastError() == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
    }
    const dim3 cgrid((ch + kCT * kCV - 1) / (kCT * kCV), a.batch, (a.L + kTT - 1) / kTT);
    if (a.bf16)
        hipLaunchKernelGGL(bdlm_conv_kernel<true>, cgrid, dim3(kCT), 0, static_cast<hipStream_t>(stream), k);
    else
        hipLaunchKernelGGL(bdlm_conv_kernel<false>, cgrid, dim3(kCT), 0, static_cast<hipStream_t>(stream), k);
    if (hipGetLastError() != hipSuccess) return BDLM_E_LAUNCH;
    if (commit) {
        hipLaunchKernelGGL(bdlm_conv_keep_kernel, dim3((ch + 255) / 256, a.batch), dim3(256), 0,
                           static_cast<hipStream_t>(stream), k);
        if (hipGetLastError() != hipSuccess) return BDLM_E_LAUNCH;
    }

    // the scan over the convolved inputs: fp32, contiguous, in the workspace
    const int64_t BL = static_cast<int64_t>(a.batch) * a.L;
    const int64_t HP = a.nheads * 64, GN = static_cast<int64_t>(a.ngroups) * a.dstate;
    float *base = static_cast<float *>(ws);
    LaunchArgs f = a, r = a;
    for (LaunchArgs *p : {&f, &r}) {
        p->bf16 = 0;
        p->xs_b = a.L * HP;
        p->xs_t = HP;
        p->xs_h = 64;
        p->dts_b = static_cast<int64_t>(a.L) * a.nheads;
        p->dts_t = a.nheads;
        p->bcs_b = a.L * GN;
        p->bcs_t = GN;
        p->bcs_g = a.dstate;
        p->dt = base + 2 * BL * (HP + 2 * GN);
    }
    f.x = base;
    f.Bm = base + BL * HP;
    f.Cm = base + BL * (HP + GN);
    r.x = base + BL * (HP + 2 * GN);
    r.Bm = base + BL * (2 * HP + 2 * GN);
    r.Cm = base + BL * (2 * HP + 3 * GN);
    // fp32 operands: both kernels contract them on fp32 MFMA
    return a.L <= BDLM_MAX_BLOCK_LEN ? launch_block_pair(f, r, commit, a.y != nullptr, stream)
                                     : launch_block_long(f, r, commit, a.y != nullptr, stream);
}

}  // namespace bdlm
