// bdlm_mask.hip -- gfx950 kernel for blocks of 65 to 256 tokens (256 is the paper's
// block length, Sec. 5.1 / App. C) in masked-matrix form: one launch computes both
// branches of Eq. partial-reverse for every token of the block and, for a commit, the
// state of Eq. boundary-state.
//
// Per (batch row b, head h), with l_t = dt_t A_h log2(e), cs_t = l_0 + ... + l_t and
// ex_t = cs_{t-1} (ex_0 = 0):
//   y[t,:] = 2^{cs_t} (C_t . s^T)                          prefix (forward only)
//          + sum_j G[t,j] W[t,j] dt_j x[j,:]                both branches at once
//          + (D + D_rev) x[t,:]
//   G[t,j] = C_t . B_j
//   W[t,j] = 2^{cs_t - cs_j} (j < t), 2 (j = t), 2^{ex_j - ex_t} (j > t)
//   s_new  = 2^{cs_{L-1}} s + sum_j 2^{cs_{L-1} - cs_j} dt_j x[j,:] (outer) B_j
// The whole block is one masked product: no chunk states, no exchange between chunks.
//
// Work split: one workgroup of eight waves per (b, h); wave w owns the output rows of
// token tiles TPW w .. TPW w + TPW - 1 (16 tokens per tile) and all 64 head-dim
// columns.  For each pair of source token tiles it forms the transposed Gram tiles
// (rows j, columns t) on bf16 MFMA from the B image in LDS and its own C quads
// (registers), weights them into the masked matrix, splits that into bf16 hi + lo and
// contracts it with x read transposed from LDS; the accumulator of the Gram product is
// already the A operand of that contraction.  The prefix term contracts the same C quads
// with the state, split once per workgroup into a bf16 hi + lo image in LDS.
//
// Decay weights off the diagonal tiles come from per-token factors relative to the
// 16-token tile boundaries (E_k = cs at the end of tile k):
//   j < t:  sLa[t] 2^{E_{mt-1} - E_jt} sLb[j],  sLa = 2^{cs_t - E_{k-1}}, sLb = 2^{E_k - cs_j} dt_j
//   j > t:  sUa[t] 2^{E_{jt-1} - E_mt} sUb[j],  sUa = 2^{E_k - ex_t},     sUb = 2^{ex_j - E_{k-1}} dt_j
// (k the token's own tile), every factor at most 1 (or dt), one exponential per tile pair;
// diagonal tiles take one exponential per element.
//
// A commit's state update contracts over tokens: B read transposed from its image,
// against the weighted x split into three bf16 terms (the new state is carried into every
// later block), starting from the cached state scaled by 2^{cs_{L-1}}.  bf16 activations.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_device.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

constexpr int kMW = 8;                 // waves per workgroup
constexpr int kMThreads = 64 * kMW;

struct MaskArgs {
    const void *x, *dt, *Bm, *Cm;      // bf16
    const float *A, *D, *D_rev;
    float *pool;                       // cached states (commit: updated in place)
    float *y;                          // outputs, or nullptr (a commit without them)
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int32_t L, nheads, heads_per_group;
    int32_t nunits;                    // (batch row, head) units
    int32_t xcd_remap;                 // units and grid % 8 == 0: a row's units on one XCD
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

constexpr uint32_t kOOB = 0x80000000u;   // offset past the resource: stores are dropped
constexpr int kNT = 2;                   // buffer cache policy: nontemporal
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             0x7fffffff, 0x00020000);
}
__device__ __forceinline__ float ex2(float v) { return __builtin_amdgcn_exp2f(v); }
__device__ __forceinline__ uint32_t lo_pair(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ __forceinline__ uint32_t hi_pair(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }
__device__ __forceinline__ f32x4 bf16x4_val(uint2 v) {
    return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                 __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u)};
}
// State quad (q, grp) of column p in the pool layout: s[p][16q + 4grp .. +3].
__device__ __forceinline__ int quad_off(int q, int grp, int p) { return ((4 * q + grp) * kP + p) * 4; }
// LDS image of B or C as 16-byte pairs of operand quads: entry (token tile mt, quad pair
// qp, lane group grp, column) holds the quads 2qp and 2qp + 1 that lane (col, grp) of an
// MFMA operand needs for rows 16mt + col (dstate 32qp + 4grp .. +3 and 32qp + 16 + 4grp ..
// +3), so one 16-byte read is a whole 32-deep operand.  The column is XOR-swizzled with
// (2qp + grp / 2) so that the 16 chunks of one row written at once land on distinct
// 16-byte slots.
template <int QP>
__device__ __forceinline__ int pair_idx(int mt, int qp, int grp, int col) {
    return (mt * QP + qp) * 64 + grp * 16 + (col ^ ((2 * qp + (grp >> 1)) & 15));
}
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
// LDS transpose read (gfx950): every lane reads four bf16 at its own 8-byte-aligned
// address, and within each group of 16 lanes, lane 4a + b receives element b of the words
// read by lanes a, a + 4, a + 8 and a + 12 of its group, in that order.
__device__ __forceinline__ s16x4 ds_read_tr(const uint2 *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(const_cast<uint2 *>(p)));
}
__device__ __forceinline__ f32x4 mma_pair(uint4 a, uint4 b, f32x4 c) {
    return mma_k32(as_s16x4(uint2{a.x, a.y}), as_s16x4(uint2{a.z, a.w}), as_s16x4(uint2{b.x, b.y}),
                   as_s16x4(uint2{b.z, b.w}), c);
}

template <int NS, int MT, bool COMMIT>
__global__ void __launch_bounds__(kMThreads) __attribute__((amdgpu_waves_per_eu(2)))
bdlm_mask_block_kernel(const MaskArgs a) {
    constexpr int QN = NS / 16;            // dstate quads
    constexpr int QP = (QN + 1) / 2;       // quad pairs (a lone last quad pairs with zeros)
    constexpr int TPW = MT / kMW;          // token tiles per wave
    constexpr int NTOK = 16 * MT;          // tokens of the padded block
    constexpr int TPL = NTOK / 64;         // tokens per lane in the decay scan
    constexpr int IMG = MT * QP * 64;      // 16-byte entries of the B or C image
    constexpr int XTQ = MT * 4 * 64;       // quads of the transposed x image
    constexpr int SQP = QP * 4 * 64;       // 16-byte entries of each state image (hi, lo)
    constexpr int REGION = IMG * 16 > XTQ * 8 + SQP * 32 ? IMG * 16 : XTQ * 8 + SQP * 32;
    constexpr int NCT = (4 * QN + kMW - 1) / kMW;   // commit tiles per wave
    static_assert(TPW >= 1 && MT % 4 == 0 && MT % kMW == 0 && (TPL == 2 || TPL == 4), "block tiles");
    // B image for the Gram tiles (and, transposed, for a commit); the region holds the C
    // image until every wave has its C quads, then the transposed x and the state's bf16 hi
    // and lo images (pairs of quads, as the B and C images)
    __shared__ __align__(16) uint4 sB[IMG];
    __shared__ __align__(16) unsigned char sU[REGION];
    __shared__ __align__(16) float sDt[NTOK], sCs[NTOK], sEx[NTOK], sEc[NTOK];
    __shared__ __align__(16) float sLa[NTOK], sLb[NTOK], sUa[NTOK], sUb[NTOK];
    __shared__ __align__(16) float sWc[COMMIT ? NTOK : 4];
    __shared__ float sE[MT];
    uint4 *sC = reinterpret_cast<uint4 *>(sU);
    uint2 *sXt = reinterpret_cast<uint2 *>(sU);
    uint4 *sSH = reinterpret_cast<uint4 *>(sU + XTQ * 8);
    uint4 *sSL = sSH + SQP;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int L = a.L;                     // 1 <= L <= NTOK
    const bool want_y = a.y != nullptr;
    const int mt0 = TPW * wave;            // first token tile of this wave's rows
    const int nunits = a.nunits;

    // One workgroup per unit (batch row, head); with the XCD remap the units of one XCD
    // (workgroup w sits on XCD w % 8) are a contiguous run, so the heads of a row share one
    // L2.
    struct Unit {
        int b, h, g;
        const uint16_t *xg, *dtg, *Bg, *Cg;
        float *hs;
    };
    auto decode = [&](int v) {
        if (a.xcd_remap) v = (v & 7) * (nunits >> 3) + (v >> 3);
        Unit un;
        un.b = v / a.nheads;
        un.h = v - un.b * a.nheads;
        un.g = un.h / a.heads_per_group;
        const int64_t slot = a.use_slots ? a.slots[un.b] : un.b;
        un.xg = static_cast<const uint16_t *>(a.x) + un.b * a.xs_b + un.h * a.xs_h;
        un.dtg = static_cast<const uint16_t *>(a.dt) + un.b * a.dts_b + un.h;
        un.Bg = static_cast<const uint16_t *>(a.Bm) + un.b * a.bcs_b + un.g * a.bcs_g;
        un.Cg = static_cast<const uint16_t *>(a.Cm) + un.b * a.bcs_b + un.g * a.bcs_g;
        un.hs = a.pool + (slot * a.nheads + un.h) * (kP * NS);
        return un;
    };
    const uint32_t bcrow = static_cast<uint32_t>(a.bcs_t * 2), xrow = static_cast<uint32_t>(a.xs_t * 2);
    const uint32_t dtrow = static_cast<uint32_t>(a.dts_t * 2);

    // ---- loads, through buffer resources with uniform bases (rows past the block get an
    // offset past the resource's range and load zeros).  B and C rows in 16-byte chunks
    // (chunk fastest: coalesced; cached, since every head of the row reads them), x in
    // four-row groups of 16-byte chunks, the state in its pool layout, dt for the scan.
    constexpr int CPR = NS / 8;                          // chunks per B / C row
    constexpr int BCN = NTOK * CPR;
    constexpr int BCK = BCN >= kMThreads ? BCN / kMThreads : 1;
    static_assert(BCN < kMThreads || BCN % kMThreads == 0, "B/C chunks");
    const bool bc_own = tid < BCN;
    constexpr int XN = 4 * MT * 8;                       // (token quad, 16-byte piece) tasks
    constexpr int XK = XN >= kMThreads ? XN / kMThreads : 1;
    static_assert(XN < kMThreads || XN % kMThreads == 0, "x tasks");
    const bool x_own = tid < XN;
    constexpr int SN = 16 * NS;                          // 16-byte chunks of one state
    constexpr int SK = SN >= kMThreads ? SN / kMThreads : 1;
    static_assert(SN < kMThreads || SN % kMThreads == 0, "state chunks");
    const bool s_own = tid < SN;
    u32x4 bch[BCK], cch[BCK], xr[XK][4], sr[SK];
    uint32_t dtraw[TPL];
    f32x4 so[NCT];
    auto load_bc = [&](const Unit &un) {
        const __amdgpu_buffer_rsrc_t rBm = rsrc(un.Bg), rCm = rsrc(un.Cg);
#pragma unroll
        for (int k = 0; k < BCK; ++k) {
            const int i = tid + kMThreads * k;
            const int t = i / CPR, c = i % CPR;
            const uint32_t o = bc_own && t < L ? t * bcrow + c * 16 : kOOB;
            bch[k] = __builtin_amdgcn_raw_buffer_load_b128(rBm, o, 0, 0);
            cch[k] = want_y ? __builtin_amdgcn_raw_buffer_load_b128(rCm, o, 0, 0) : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto load_rest = [&](const Unit &un) {
        const __amdgpu_buffer_rsrc_t rX = rsrc(un.xg), rD = rsrc(un.dtg), rS = rsrc(un.hs);
#pragma unroll
        for (int i = 0; i < TPL; ++i) {
            const int t = TPL * lane + i;
            dtraw[i] = __builtin_amdgcn_raw_buffer_load_b16(rD, t < L ? t * dtrow : kOOB, 0, 0);
        }
#pragma unroll
        for (int k = 0; k < XK; ++k) {
            const int task = tid + kMThreads * k;
            const int tq = task >> 3, pc = task & 7;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 4 * tq + r;
                xr[k][r] = __builtin_amdgcn_raw_buffer_load_b128(rX, x_own && t < L ? t * xrow + pc * 16 : kOOB, 0, kNT);
            }
        }
#pragma unroll
        for (int k = 0; k < SK; ++k) {
            const uint32_t o = want_y && s_own ? 16u * (tid + kMThreads * k) : kOOB;
            sr[k] = __builtin_amdgcn_raw_buffer_load_b128(rS, o, 0, kNT);
        }
        // a commit's own tiles of the state (tile k = wave + 8i: columns 16 (k & 3) .., quad k >> 2)
        if constexpr (COMMIT) {
#pragma unroll
            for (int i = 0; i < NCT; ++i) {
                const int k = wave + kMW * i;
                const uint32_t o = k < 4 * QN ? 4u * quad_off(k >> 2, grp, 16 * (k & 3) + col) : kOOB;
                so[i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rS, o, 0, 0));
            }
        }
    };

    const int unit = blockIdx.x;
    if (unit >= nunits) return;
    const Unit un = decode(unit);
    load_bc(un);
    load_rest(un);
    {

        // ---- B and C images; the decay sums (wave 0, TPL tokens per lane)
        {
            uint2 *b2 = reinterpret_cast<uint2 *>(sB), *c2 = reinterpret_cast<uint2 *>(sC);
#pragma unroll
            for (int k = 0; k < BCK; ++k) {
                if (!bc_own) break;
                const int i = tid + kMThreads * k;
                const int t = i / CPR, c = i % CPR;
                // 8 bf16 = quad q = c / 2 of lane groups 2 (c % 2) and 2 (c % 2) + 1
                const int q = c >> 1, gr = 2 * (c & 1);
                const int at = 2 * pair_idx<QP>(t >> 4, q >> 1, gr, t & 15) + (q & 1);
                const int at1 = 2 * pair_idx<QP>(t >> 4, q >> 1, gr + 1, t & 15) + (q & 1);
                b2[at] = uint2{bch[k].x, bch[k].y};
                b2[at1] = uint2{bch[k].z, bch[k].w};
                if constexpr (QN & 1) {   // the lone last quad's partner is zero
                    if (q == QN - 1) b2[at + 1] = b2[at1 + 1] = uint2{0u, 0u};
                }
                if (want_y) {
                    c2[at] = uint2{cch[k].x, cch[k].y};
                    c2[at1] = uint2{cch[k].z, cch[k].w};
                    if constexpr (QN & 1) {
                        if (q == QN - 1) c2[at + 1] = c2[at1 + 1] = uint2{0u, 0u};
                    }
                }
            }
        }
        if (wave == 0) {
            const float A2 = a.A[un.h] * kLog2e;
            float dtv[TPL], cs[TPL], ex[TPL];
            float run = 0.f;
#pragma unroll
            for (int i = 0; i < TPL; ++i) {
                dtv[i] = __uint_as_float(dtraw[i] << 16);
                run += dtv[i] * A2;
                cs[i] = run;
            }
            const float incl = wave_inclusive_sum(run);
            const float up = __shfl_up(incl, 1, 64);
            const float excl = lane == 0 ? 0.f : up;
#pragma unroll
            for (int i = 0; i < TPL; ++i) cs[i] += excl;
            const float prev = __shfl_up(cs[TPL - 1], 1, 64);
            ex[0] = lane == 0 ? 0.f : prev;
#pragma unroll
            for (int i = 1; i < TPL; ++i) ex[i] = cs[i - 1];
            // this lane's tile k; E_k and E_{k-1} from the lanes holding tokens 16k + 15, 16k - 1
            const int k = (TPL * lane) >> 4;
            constexpr int LPT = 16 / TPL;      // lanes per tile
            const float Ek = __shfl(cs[TPL - 1], LPT * k + LPT - 1, 64);
            const float Ekm = __shfl(cs[TPL - 1], k > 0 ? LPT * k - 1 : 0, 64);
            const float Ekm1 = k > 0 ? Ekm : 0.f;
            const float Elast = __shfl(cs[TPL - 1], 63, 64);
#pragma unroll
            for (int i = 0; i < TPL; ++i) {
                const int t = TPL * lane + i;
                sDt[t] = dtv[i];
                sCs[t] = cs[i];
                sEx[t] = ex[i];
                sEc[t] = ex2(cs[i]);
                sLa[t] = ex2(cs[i] - Ekm1);
                sLb[t] = ex2(Ek - cs[i]) * dtv[i];
                sUa[t] = ex2(Ek - ex[i]);
                sUb[t] = ex2(ex[i] - Ekm1) * dtv[i];
                if constexpr (COMMIT) sWc[t] = ex2(Elast - cs[i]) * dtv[i];
            }
            if ((lane & (LPT - 1)) == LPT - 1) sE[k] = cs[TPL - 1];
        }
        __syncthreads();

        // ---- this wave's C quad pairs (rows 16 mt + col): the B operand of its Gram tiles
        // and the A operand of its prefix terms
        uint4 cq[TPW][QP];
        if (want_y) {
#pragma unroll
            for (int m = 0; m < TPW; ++m)
#pragma unroll
                for (int qp = 0; qp < QP; ++qp) cq[m][qp] = sC[pair_idx<QP>(mt0 + m, qp, grp, col)];
            __syncthreads();   // the C image is overwritten next
        }

        // ---- transposed x (quad (token quad tq, column p): tokens 4tq .. 4tq+3) and the
        // state split into bf16 hi + lo (entry (quad pair, lane group, column): quads 2qp,
        // 2qp + 1)
#pragma unroll
        for (int k = 0; k < XK; ++k) {
            if (!x_own) break;
            const int task = tid + kMThreads * k;
            const int tq = task >> 3, pc = task & 7;
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                sXt[tq * kP + pc * 8 + 2 * d] = uint2{lo_pair(xr[k][0][d], xr[k][1][d]), lo_pair(xr[k][2][d], xr[k][3][d])};
                sXt[tq * kP + pc * 8 + 2 * d + 1] = uint2{hi_pair(xr[k][0][d], xr[k][1][d]), hi_pair(xr[k][2][d], xr[k][3][d])};
            }
        }
        if (want_y) {
            uint2 *sh2 = reinterpret_cast<uint2 *>(sSH), *sl2 = reinterpret_cast<uint2 *>(sSL);
#pragma unroll
            for (int k = 0; k < SK; ++k) {
                if (!s_own) break;
                const int i = tid + kMThreads * k;             // pool-layout chunk (4q + grp) * 64 + p
                const int q = i >> 8, gp = i & 255;             // gp = grp * 64 + p
                s16x4 hi, lo;
                split4(__builtin_bit_cast(f32x4, sr[k]), hi, lo);
                const int at = 2 * ((q >> 1) * 256 + gp) + (q & 1);
                sh2[at] = as_u2(hi);
                sl2[at] = as_u2(lo);
                if constexpr (QN & 1) {
                    if (q == QN - 1) sh2[at + 1] = sl2[at + 1] = uint2{0u, 0u};
                }
            }
        }
        const int hcur = un.h, bcur = un.b;
        float *const hs_cur = un.hs;
        __syncthreads();

        if (want_y) {
            // ---- masked product: rows t of this wave's tiles, sources j over the block
            f32x4 Y[TPW][4];
#pragma unroll
            for (int m = 0; m < TPW; ++m)
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) Y[m][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
            float la[TPW], ua[TPW];
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                const int t = 16 * (mt0 + m) + col;
                la[m] = sLa[t];
                ua[m] = sUa[t];
            }
            // the tile-pair factors of this wave's rows, lane m MT + jt: 2^{E_{mt-1} - E_jt}
            // below the diagonal, 2^{E_{jt-1} - E_mt} above it, 0 on it (the diagonal tiles
            // follow the loop)
            float tf;
            {
                const int m = lane / MT, jt = lane % MT;
                const int mt = mt0 + (m < TPW ? m : 0);
                const bool below = lane < TPW * MT && jt < mt, above = lane < TPW * MT && jt > mt;
                const float e = below ? sE[mt > 0 ? mt - 1 : 0] - sE[jt]
                                      : sE[jt > 0 ? jt - 1 : 0] - sE[mt];
                tf = below || above ? ex2(e) : 0.f;
            }
            // Gram tiles of source tiles j0, j0 + 1, transposed: lane (col, grp) holds G[t][j],
            // t = 16 mt + col, j = 16 jt + 4 grp + r
            auto gram = [&](int j0, f32x4 (&gt)[2][TPW]) {
#pragma unroll
                for (int d = 0; d < 2; ++d) {
                    uint4 bj[QP];
#pragma unroll
                    for (int qp = 0; qp < QP; ++qp) bj[qp] = sB[pair_idx<QP>(j0 + d, qp, grp, col)];
#pragma unroll
                    for (int m = 0; m < TPW; ++m) {
                        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int qp = 0; qp < QP; ++qp) acc = mma_pair(bj[qp], cq[m][qp], acc);
                        gt[d][m] = acc;
                    }
                }
            };
            // weighted and split (the A operands of the two source tiles side by side), then
            // contracted with x
            auto consume = [&](int j0, const f32x4 (&gt)[2][TPW]) {
                uint4 mh[TPW], ml[TPW];
#pragma unroll
                for (int m = 0; m < TPW; ++m) {
                    const int mt = mt0 + m;
                    uint2 hh[2], ll[2];
#pragma unroll
                    for (int d = 0; d < 2; ++d) {
                        const int jt = j0 + d;
                        const bool below = jt < mt;
                        const float sf = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(tf), m * MT + jt));
                        const float f = (below ? la[m] : ua[m]) * sf;
                        const f32x4 fac = *reinterpret_cast<const f32x4 *>((below ? sLb : sUb) + 16 * jt + 4 * grp);
                        s16x4 th, tl;
                        split4(gt[d][m] * (fac * f), th, tl);
                        hh[d] = as_u2(th);
                        ll[d] = as_u2(tl);
                    }
                    mh[m] = uint4{hh[0].x, hh[0].y, hh[1].x, hh[1].y};
                    ml[m] = uint4{ll[0].x, ll[0].y, ll[1].x, ll[1].y};
                }
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    const uint2 x0 = sXt[(4 * j0 + grp) * kP + 16 * pt + col];
                    const uint2 x1 = sXt[(4 * (j0 + 1) + grp) * kP + 16 * pt + col];
                    const uint4 xq = uint4{x0.x, x0.y, x1.x, x1.y};
#pragma unroll
                    for (int m = 0; m < TPW; ++m) {
                        Y[m][pt] = mma_pair(mh[m], xq, Y[m][pt]);
                        Y[m][pt] = mma_pair(ml[m], xq, Y[m][pt]);
                    }
                }
            };
            // two pairs of source tiles per iteration: the next pair's Gram products are
            // issued before this pair's weights are computed, so matrix and vector work overlap
            f32x4 ga[2][TPW], gb[2][TPW];
            gram(0, ga);
#pragma unroll 1
            for (int j0 = 0; j0 < MT; j0 += 4) {
                gram(j0 + 2, gb);
                consume(j0, ga);
                if (j0 + 4 < MT) gram(j0 + 4, ga);
                consume(j0 + 2, gb);
            }
            // the diagonal tiles: both branches, and the token's own input twice
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                const int mt = mt0 + m;
                f32x4 gd = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int qp = 0; qp < QP; ++qp) gd = mma_pair(sB[pair_idx<QP>(mt, qp, grp, col)], cq[m][qp], gd);
                const float cst = sCs[16 * mt + col], ext = sEx[16 * mt + col];
                const f32x4 csj = *reinterpret_cast<const f32x4 *>(&sCs[16 * mt + 4 * grp]);
                const f32x4 exj = *reinterpret_cast<const f32x4 *>(&sEx[16 * mt + 4 * grp]);
                const f32x4 dtj = *reinterpret_cast<const f32x4 *>(&sDt[16 * mt + 4 * grp]);
                f32x4 w;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int j = 4 * grp + r;   // positions within the tile
                    const float e = ex2(j < col ? cst - csj[r] : exj[r] - ext);
                    w[r] = (j == col ? 2.f : e) * dtj[r];
                }
                s16x4 th, tl;
                split4(gd * w, th, tl);
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    const s16x4 xq = as_s16x4(sXt[(4 * mt + grp) * kP + 16 * pt + col]);
                    // Y comes from 32-deep MFMAs: stay on that shape (zero upper half)
                    constexpr s16x4 z = {0, 0, 0, 0};
                    Y[m][pt] = mma_k32(th, z, xq, z, Y[m][pt]);
                    Y[m][pt] = mma_k32(tl, z, xq, z, Y[m][pt]);
                }
            }

            // ---- prefix term 2^{cs_t} (C_t . s^T), skip term, store (lane (col, grp): token
            // 16 mt + 4 grp + r, column 16 pt + col); tokens past the block are dropped
            const float skip = a.D[hcur] + a.D_rev[hcur];
            const __amdgpu_buffer_rsrc_t rY =
                rsrc(a.y + ((static_cast<int64_t>(bcur) * L) * a.nheads + hcur) * kP);   // uniform base
            const uint32_t ytokB = static_cast<uint32_t>(a.nheads) * kP * 4;
            uint32_t yo[TPW][4];
            f32x4 ec[TPW];
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                ec[m] = *reinterpret_cast<const f32x4 *>(&sEc[16 * (mt0 + m) + 4 * grp]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * (mt0 + m) + 4 * grp + r;
                    yo[m][r] = t < L ? t * ytokB + 4 * col : kOOB;
                }
            }
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
                f32x4 Z[TPW];
#pragma unroll
                for (int m = 0; m < TPW; ++m) Z[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int qp = 0; qp < QP; ++qp) {
                    const uint4 sh = sSH[(qp * 4 + grp) * kP + 16 * pt + col];
                    const uint4 sl = sSL[(qp * 4 + grp) * kP + 16 * pt + col];
#pragma unroll
                    for (int m = 0; m < TPW; ++m) {
                        Z[m] = mma_pair(cq[m][qp], sh, Z[m]);
                        Z[m] = mma_pair(cq[m][qp], sl, Z[m]);
                    }
                }
#pragma unroll
                for (int m = 0; m < TPW; ++m) {
                    const f32x4 xv = bf16x4_val(sXt[(4 * (mt0 + m) + grp) * kP + 16 * pt + col]);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float out = ec[m][r] * Z[m][r] + Y[m][pt][r] + skip * xv[r];
                        // through the cache: a row's four 64-byte pieces (pt) meet in L2
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(out), rY, yo[m][r], 64 * pt, 0);
                    }
                }
            }
        }

        if constexpr (COMMIT) {
            // ---- s_new[p, n] = 2^{cs_last} s[p, n] + sum_j B[j, n] wc_j x[j, p] on this
            // wave's tiles (columns 16 pt + col, pt = wave & 3 for every tile of the wave).
            // A operand: lane (col, grp) holds B[16 jt + 4 grp + r][16 q + col], read
            // transposed from the B image.
            const float keep = ex2(sE[MT - 1]);
            const int pt = wave & 3;
            uint2 wh[MT], wm[MT], wl[MT];
#pragma unroll
            for (int jt = 0; jt < MT; ++jt) {
                const f32x4 wc = *reinterpret_cast<const f32x4 *>(&sWc[16 * jt + 4 * grp]);
                const f32x4 xv = bf16x4_val(sXt[(4 * jt + grp) * kP + 16 * pt + col]);
                s16x4 th, tm, tl;
                split4x3(wc * xv, th, tm, tl);
                wh[jt] = as_u2(th);
                wm[jt] = as_u2(tm);
                wl[jt] = as_u2(tl);
            }
            const uint2 *sB2 = reinterpret_cast<const uint2 *>(sB);
            // the quad this lane reads for the transposed operand: token 16 jt + tt, dstate
            // 16 q + 4 (lane % 4) .. +3 (lane group lane % 4 of the B image)
            const int tt = 4 * (lane >> 4) + ((lane & 15) >> 2), ta = lane & 3;
#pragma unroll
            for (int i = 0; i < NCT; ++i) {
                const int k = wave + kMW * i;
                if (k >= 4 * QN) break;
                const int q = k >> 2;
                f32x4 acc = so[i] * keep;
#pragma unroll
                for (int jt = 0; jt < MT; jt += 2) {
                    // B[16 (jt + d) + 4 grp + r][16 q + col], r = 0 .. 3, through the LDS
                    // transpose read (one 8-byte read per lane)
                    const s16x4 b0 = ds_read_tr(sB2 + 2 * pair_idx<QP>(jt, q >> 1, ta, tt) + (q & 1));
                    const s16x4 b1 = ds_read_tr(sB2 + 2 * pair_idx<QP>(jt + 1, q >> 1, ta, tt) + (q & 1));
                    acc = mma_k32(b0, b1, as_s16x4(wh[jt]), as_s16x4(wh[jt + 1]), acc);
                    acc = mma_k32(b0, b1, as_s16x4(wm[jt]), as_s16x4(wm[jt + 1]), acc);
                    acc = mma_k32(b0, b1, as_s16x4(wl[jt]), as_s16x4(wl[jt + 1]), acc);
                }
                *reinterpret_cast<f32x4 *>(hs_cur + quad_off(q, grp, 16 * pt + col)) = acc;
            }
        }
    }
}

template <int NS, int MT>
hipError_t mask_launch(const MaskArgs &k, bool commit, unsigned grid, hipStream_t s) {
    if (commit)
        hipLaunchKernelGGL((bdlm_mask_block_kernel<NS, MT, true>), dim3(grid), dim3(kMThreads), 0, s, k);
    else
        hipLaunchKernelGGL((bdlm_mask_block_kernel<NS, MT, false>), dim3(grid), dim3(kMThreads), 0, s, k);
    return hipGetLastError();
}
template <int NS>
hipError_t mask_mt(const MaskArgs &k, int L, bool commit, unsigned grid, hipStream_t s) {
    return L <= 128 ? mask_launch<NS, 8>(k, commit, grid, s) : mask_launch<NS, 16>(k, commit, grid, s);
}

}  // namespace

bool long_masked_fits(const LaunchArgs &a) {
    return a.bf16 && a.L > 64 && a.L <= 256 && a.batch <= BDLM_MAX_SLOT_ROWS &&
           (a.dstate == 16 || a.dstate == 32 || a.dstate == 64 || a.dstate == 128);
}

int launch_block_long_shared(const LaunchArgs &a, bool commit, bool want_y, void *stream) {
    return long_masked_fits(a) ? launch_long_masked(a, commit, want_y, stream)
                               : launch_block_long(a, a, commit, want_y, stream);
}

int launch_long_masked(const LaunchArgs &a, bool commit, bool want_y, void *stream) {
    if (a.batch == 0 || a.L == 0) return BDLM_OK;
    if (!long_masked_fits(a)) return BDLM_E_SHAPE;
    if (!commit && !want_y) return BDLM_OK;
    MaskArgs k;
    k.x = a.x;
    k.dt = a.dt;
    k.Bm = a.Bm;
    k.Cm = a.Cm;
    k.A = a.A;
    k.D = a.D;
    k.D_rev = a.D_rev;
    k.pool = a.h_pool;
    k.y = want_y ? a.y : nullptr;
    k.xs_b = a.xs_b;
    k.xs_t = a.xs_t;
    k.xs_h = a.xs_h;
    k.dts_b = a.dts_b;
    k.dts_t = a.dts_t;
    k.bcs_b = a.bcs_b;
    k.bcs_t = a.bcs_t;
    k.bcs_g = a.bcs_g;
    k.L = a.L;
    k.nheads = a.nheads;
    k.heads_per_group = a.nheads / a.ngroups;
    k.use_slots = a.slots ? 1 : 0;
    for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i) k.slots[i] = (a.slots && i < a.batch) ? a.slots[i] : 0;
    const int64_t units = static_cast<int64_t>(a.batch) * a.nheads;
    const int64_t grid = units;
    k.nunits = static_cast<int32_t>(units);
    k.xcd_remap = units % 8 == 0 ? 1 : 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const unsigned gr = static_cast<unsigned>(grid);
    hipError_t e;
    switch (a.dstate) {
        case 16: e = mask_mt<16>(k, a.L, commit, gr, s); break;
        case 32: e = mask_mt<32>(k, a.L, commit, gr, s); break;
        case 64: e = mask_mt<64>(k, a.L, commit, gr, s); break;
        default: e = mask_mt<128>(k, a.L, commit, gr, s); break;
    }
    return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

}  // namespace bdlm
