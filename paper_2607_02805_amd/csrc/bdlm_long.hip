// bdlm_long.hip -- gfx950 kernel for blocks of 65 to 256 tokens (256 is the paper's
// block length, Sec. 5.1 / App. C): one launch computes both branches of Eq.
// partial-reverse for every token of the block and, for a commit, the state of Eq.
// boundary-state, with the block's 64-token chunks processed side by side instead of
// one after the other.
//
// Chunk decomposition.  The block is cut into NCH chunks of 64 tokens; wave c of a
// workgroup owns chunk c.  Within a chunk, with l_i = dt_i A_h log2(e), cs the
// inclusive sums from the chunk start, ex_i = cs_{i-1} (ex_0 = 0) and tot = cs_63:
//   forward   h_t = 2^{cs_t} S_c + sum_{j<=t} 2^{cs_t - cs_j} dt_j x_j B_j
//             S_0 = the cached state,  S_{c+1} = 2^{tot_c} S_c + F_c,
//             F_c = sum_j 2^{tot_c - cs_j} dt_j x_j B_j           (local forward state)
//   reverse   g_t = 2^{tot_c - ex_t} E_c + sum_{j>=t} 2^{ex_j - ex_t} dt_j x_j B_j
//             E_c = R_{c+1} + 2^{tot_{c+1}} E_{c+1},  E_{NCH-1} = 0,
//             R_k = sum_j 2^{ex_j} dt_j x_j B_j                     (local reverse state)
//   y_t = C_t . (h_t + g_t) + (D + D_rev) x_t
// (the reverse decay from j to t < j is a_t ... a_{j-1}, as in the block kernel).  Each
// wave computes its chunk's local states, publishes them in LDS, and after one barrier
// assembles S_c and E_c from the other chunks' states; the intra-chunk terms of both
// branches are one masked product with 2 dt_t on the diagonal.  A commit's new state is
// 2^{tot} S_{NCH-1} + F_{NCH-1}, written by the last chunk's wave.
//
// Work split: one workgroup per (batch row, head, 16 head-dim columns), so a state
// slice (16 x N) fits one wave's registers and the grid holds four workgroups per
// (row, head).  Every wave computes its chunk's full decay-weighted Gram matrix C.B^T
// (the four column slices of a head each recompute it) on bf16 MFMA.  B and C are
// loaded as whole rows (every 16 lanes read 256 contiguous bytes) and rearranged into
// operand quads through a row image in the wave's own LDS region: C's quads are kept in
// registers for the Gram tiles and the prefix terms, B's are read back for the Gram
// tiles and, transposed, for the contractions over tokens (local states); the region
// then holds the local states the wave publishes.  Decay weights come from per-token
// factors relative to 16-token tile boundaries (one exponential per token and factor,
// one per tile pair), each at most 1.  Products with an fp32 operand split it into bf16
// terms (two; three for the local forward states of a commit, whose sum becomes a
// cached state).  bf16 activations only.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_device.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

constexpr int kCh = 64;               // tokens per chunk (one per lane in the decay scan)
constexpr int kPS = 16;               // head-dim columns per workgroup
constexpr int kSlices = kP / kPS;     // workgroups per (row, head)

struct LongArgs {
    const void *x, *dt, *Bm, *Cm;     // bf16
    const float *A, *D, *D_rev;
    float *pool;                      // cached states (commit: updated in place)
    float *y;                         // outputs, or nullptr (a commit without them)
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int32_t L, nheads, heads_per_group;
    int32_t xcd_remap;                // grid % 8 == 0: a row's workgroups on one XCD
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

constexpr uint32_t kOOB = 0x80000000u;   // offset past the resource: loads read zero
constexpr int kNT = 2;                   // buffer cache policy: nontemporal
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             0x7fffffff, 0x00020000);
}
__device__ __forceinline__ float ex2(float v) { return __builtin_amdgcn_exp2f(v); }
// 8-byte load at per-lane offset vo plus uniform offset so (an out-of-range vo stays out
// of range)
__device__ __forceinline__ uint2 ld64(__amdgpu_buffer_rsrc_t r, uint32_t vo, uint32_t so) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, vo, so, 0);
    return uint2{v[0], v[1]};
}
__device__ __forceinline__ f32x4 bf16x4_val(uint2 v) {
    return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                 __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u)};
}
// c += A B over Q operand quads (16 contraction indices each), pairs on the 32-deep
// instruction
template <int Q>
__device__ __forceinline__ f32x4 mma_q(const uint2 *a, const uint2 *b, f32x4 c) {
#pragma unroll
    for (int q = 0; q + 1 < Q; q += 2)
        c = mma_k32(as_s16x4(a[q]), as_s16x4(a[q + 1]), as_s16x4(b[q]), as_s16x4(b[q + 1]), c);
    if constexpr (Q & 1) c = mma_k16(as_s16x4(a[Q - 1]), as_s16x4(b[Q - 1]), c);
    return c;
}
// The fp32 operand of a product as bf16 terms: hi + lo, or hi + mid + lo (T3).
template <bool T3> struct Terms { uint2 h, m, l; };
template <bool T3>
__device__ __forceinline__ Terms<T3> terms(f32x4 v) {
    Terms<T3> t;
    s16x4 h, m, l;
    if constexpr (T3) split4x3(v, h, m, l);
    else {
        split4(v, h, l);
        m = s16x4{0, 0, 0, 0};
    }
    t.h = as_u2(h);
    t.m = as_u2(m);
    t.l = as_u2(l);
    return t;
}
// c += A (bf16, exact) times the four token quads of W (split into terms)
template <bool T3>
__device__ __forceinline__ f32x4 mma_w(const uint2 (&a)[4], const Terms<T3> (&w)[4], f32x4 c) {
#pragma unroll
    for (int jt = 0; jt < 4; jt += 2) {
        const s16x4 a0 = as_s16x4(a[jt]), a1 = as_s16x4(a[jt + 1]);
        c = mma_k32(a0, a1, as_s16x4(w[jt].h), as_s16x4(w[jt + 1].h), c);
        if constexpr (T3) c = mma_k32(a0, a1, as_s16x4(w[jt].m), as_s16x4(w[jt + 1].m), c);
        c = mma_k32(a0, a1, as_s16x4(w[jt].l), as_s16x4(w[jt + 1].l), c);
    }
    return c;
}

// State quad (q, grp) of column p in the pool layout: s[p][16q + 4grp .. +3].
__device__ __forceinline__ int quad_off(int q, int grp, int p) { return ((4 * q + grp) * kP + p) * 4; }

template <int NS, int NCH, bool COMMIT>
__global__ void __launch_bounds__(64 * NCH) __attribute__((amdgpu_waves_per_eu(2)))
bdlm_long_block_kernel(const LongArgs a) {
    constexpr int QN = NS / 16;        // dstate quads
    // row stride (elements) of a wave's row images: NS + 8 puts consecutive rows 4 banks
    // apart, so the operand-quad reads (16 rows x 4 lane groups), the transposed two-byte
    // reads and the 16-byte row writes spread over the banks (measured: no conflicts left
    // but those of the two-byte reads themselves)
    constexpr int RS = NS + 8;
    constexpr int REG = kCh * RS * 2;  // bytes of a wave's LDS region
    constexpr int PR = NS / 8;         // 16-byte pieces per B / C row
    constexpr int RPI = 64 / PR;       // rows per load instruction (a row per PR lanes)
    static_assert(REG >= 2 * QN * 64 * 16, "the region holds both local states");
    // a wave's region: its chunk's C rows, then its B rows (element (j, n) at j * RS + n),
    // then the local states it publishes (forward quads, then reverse quads,
    // (4q + grp) * 16 + col)
    __shared__ __align__(16) unsigned char sReg[NCH][REG];
    // per token t of each chunk (lane t of its wave): decay sums, dt, and the decay factors
    // the products use (tile k = tokens 16k .. 16k+15, E_k = cs at the end of tile k, X_k =
    // ex at its start; every factor is at most 1, or dt):
    //   sEc = 2^{cs_t}, sEr = 2^{tot - ex_t}          prefix terms (forward, reverse)
    //   sWf = 2^{tot - cs_t} dt_t, sWr = 2^{ex_t} dt_t  local states (forward, reverse)
    //   sLa = 2^{cs_t - E_{k-1}}, sLb = 2^{E_k - cs_t} dt_t       below-diagonal tiles
    //   sUa = 2^{X_{k+1} - ex_t}, sUb = 2^{ex_t - X_k} dt_t       above-diagonal tiles
    // (k the tile of t), so the weight of source j in tile jt on target t in tile mt is
    // sLa[t] 2^{E_{mt-1} - E_jt} sLb[j] below the diagonal and sUa[t] 2^{X_jt - X_{mt+1}}
    // sUb[j] above it, with one exponential per tile pair; diagonal tiles use cs, ex, dt.
    __shared__ __align__(16) float sCs[NCH][kCh], sEx[NCH][kCh], sDt[NCH][kCh];
    __shared__ __align__(16) float sEc[NCH][kCh], sEr[NCH][kCh], sWf[NCH][kCh], sWr[NCH][kCh];
    __shared__ __align__(16) float sLa[NCH][kCh], sLb[NCH][kCh], sUa[NCH][kCh], sUb[NCH][kCh];
    __shared__ float sTot[NCH];

    const int lane = threadIdx.x & 63;
    const int c = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);   // chunk
    const int col = lane & 15, grp = lane >> 4;
    int u = blockIdx.x;
    if (a.xcd_remap) u = (u & 7) * (static_cast<int>(gridDim.x) >> 3) + (u >> 3);
    const int sl = u % kSlices;
    const int rest = u / kSlices;
    const int h = rest % a.nheads, b = rest / a.nheads;
    const int g = h / a.heads_per_group;
    const int p0 = kPS * sl, p = p0 + col;
    const int t0 = kCh * c;
    const int lim = a.L - t0 < kCh ? a.L - t0 : kCh;   // valid tokens of this chunk (>= 1)
    const bool want_y = a.y != nullptr;
    uint16_t *img = reinterpret_cast<uint16_t *>(sReg[c]);

    // ---- loads: dt (lane = token), B and C rows, x quads (tokens 16jt + 4grp .. +3 at
    // column p); rows past the block read 0 (resource bases are uniform across the wave: a
    // per-lane base would make the compiler loop over the lanes' distinct values for every
    // access)
    const char *xb = static_cast<const char *>(a.x) + (b * a.xs_b + t0 * a.xs_t + h * a.xs_h + p0) * 2;
    const char *db = static_cast<const char *>(a.dt) + (b * a.dts_b + t0 * a.dts_t + h) * 2;
    const int64_t bco = (b * a.bcs_b + t0 * a.bcs_t + g * a.bcs_g) * 2;
    const __amdgpu_buffer_rsrc_t rX = rsrc(xb), rD = rsrc(db);
    const __amdgpu_buffer_rsrc_t rB = rsrc(static_cast<const char *>(a.Bm) + bco);
    const __amdgpu_buffer_rsrc_t rC = rsrc(static_cast<const char *>(a.Cm) + bco);
    const uint32_t xrow = static_cast<uint32_t>(a.xs_t * 2), bcrow = static_cast<uint32_t>(a.bcs_t * 2);

    const uint32_t dtraw = __builtin_amdgcn_raw_buffer_load_b16(
        rD, lane < lim ? static_cast<uint32_t>(lane * a.dts_t * 2) : kOOB, 0, 0);
    // B and C rows: PR consecutive lanes read one 16-byte piece each of a row, so every
    // group of 16 lanes reads contiguous memory (the MFMA operand layout, a row per lane,
    // would touch 16 rows per 16 lanes); the wave rearranges them through LDS
    u32x4 braw[PR], craw[PR];
    {
        const int rl = lane / PR, pc = lane % PR;
#pragma unroll
        for (int i = 0; i < PR; ++i) {
            const int row = RPI * i + rl;
            const uint32_t o = row < lim ? row * bcrow + pc * 16 : kOOB;
            if (want_y) craw[i] = __builtin_amdgcn_raw_buffer_load_b128(rC, o, 0, 0);
            braw[i] = __builtin_amdgcn_raw_buffer_load_b128(rB, o, 0, 0);
        }
    }
    auto stage_rows = [&](const u32x4 (&v)[PR]) {
        const int rl = lane / PR, pc = lane % PR;
#pragma unroll
        for (int i = 0; i < PR; ++i)
            *reinterpret_cast<u32x4 *>(&img[(RPI * i + rl) * RS + pc * 8]) = v[i];
    };
    uint2 xq[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        uint32_t v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int j = 16 * jt + 4 * grp + r;
            v[r] = __builtin_amdgcn_raw_buffer_load_b16(rX, j < lim ? j * xrow + 2 * col : kOOB, 0, 0);
        }
        xq[jt] = uint2{v[0] | (v[1] << 16), v[2] | (v[3] << 16)};
    }

    // ---- decay sums of the chunk (base 2)
    const float A2 = a.A[h] * kLog2e;
    const float dtv = __uint_as_float(dtraw << 16);
    const float cs = wave_inclusive_sum(dtv * A2);
    const float up = __shfl_up(cs, 1, 64);
    const float tot = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cs), 63));
    const float ex = lane == 0 ? 0.f : up;
    // tile boundaries (uniform): E_k = cs at token 16k + 15, X_k = ex at token 16k = E_{k-1}
    float Eb[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) Eb[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cs), 16 * k + 15));
    auto Xb = [&](int k) { return k == 0 ? 0.f : Eb[k - 1]; };
    {
        const int k = lane >> 4;
        const float Ekm1 = k == 0 ? 0.f : (k == 1 ? Eb[0] : (k == 2 ? Eb[1] : Eb[2]));
        const float Ek = k == 0 ? Eb[0] : (k == 1 ? Eb[1] : (k == 2 ? Eb[2] : Eb[3]));
        const float Xk1 = Ek;   // X_{k+1} = E_k
        const float Xk = Ekm1;  // X_k = E_{k-1}
        sCs[c][lane] = cs;
        sEx[c][lane] = ex;
        sDt[c][lane] = dtv;
        sEc[c][lane] = ex2(cs);
        sEr[c][lane] = ex2(tot - ex);
        sWf[c][lane] = ex2(tot - cs) * dtv;
        sWr[c][lane] = ex2(ex) * dtv;
        sLa[c][lane] = ex2(cs - Ekm1);
        sLb[c][lane] = ex2(Ek - cs) * dtv;
        sUa[c][lane] = ex2(Xk1 - ex);
        sUb[c][lane] = ex2(ex - Xk) * dtv;
    }
    if (lane == 0) sTot[c] = tot;

    // ---- C operand quads (row 16mt + col, dstate 16q + 4grp .. +3) from a row image, kept
    // in registers for the Gram tiles and the prefix terms; then the B row image
    uint2 cq[4][QN];
    if (want_y) {
        stage_rows(craw);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int q = 0; q < QN; ++q)
                cq[mt][q] = *reinterpret_cast<const uint2 *>(&img[(16 * mt + col) * RS + 16 * q + 4 * grp]);
    }
    stage_rows(braw);

    f32x4 Y[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) Y[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the wave's own LDS writes are complete before it reads them back
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");

    if (want_y) {
        // ---- decay-weighted Gram tiles, transposed (lane (col, grp): j = 16jt + 4grp + r,
        // t = 16mt + col), weighted as the masked matrix of both branches, and the
        // intra-chunk product y[t] += sum_j M[t][j] x[j]
        float cst[4], ext[4], lat[4], uat[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            cst[mt] = sCs[c][16 * mt + col];
            ext[mt] = sEx[c][16 * mt + col];
            lat[mt] = sLa[c][16 * mt + col];
            uat[mt] = sUa[c][16 * mt + col];
        }
#pragma unroll
        for (int jt = 0; jt < 4; jt += 2) {
            uint2 mh[2][4], ml[2][4];
            // the eight tiles of token tiles jt, jt + 1 side by side (independent
            // accumulations interleave on the matrix unit)
            f32x4 gacc[2][4];
            {
                uint2 bj[2][QN];   // B operand quads, read back from the row image
#pragma unroll
                for (int d = 0; d < 2; ++d)
#pragma unroll
                    for (int q = 0; q < QN; ++q)
                        bj[d][q] = *reinterpret_cast<const uint2 *>(
                            &img[(16 * (jt + d) + col) * RS + 16 * q + 4 * grp]);
#pragma unroll
                for (int d = 0; d < 2; ++d)
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt) gacc[d][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < QN; q += 2)
#pragma unroll
                    for (int d = 0; d < 2; ++d)
#pragma unroll
                        for (int mt = 0; mt < 4; ++mt) {
                            if constexpr (QN == 1)
                                gacc[d][mt] = mma_k16(as_s16x4(bj[d][0]), as_s16x4(cq[mt][0]), gacc[d][mt]);
                            else
                                gacc[d][mt] = mma_k32(as_s16x4(bj[d][q]), as_s16x4(bj[d][q + 1]),
                                                      as_s16x4(cq[mt][q]), as_s16x4(cq[mt][q + 1]),
                                                      gacc[d][mt]);
                        }
            }
#pragma unroll
            for (int d = 0; d < 2; ++d) {
                const int jj = jt + d;
                const f32x4 lbj = *reinterpret_cast<const f32x4 *>(&sLb[c][16 * jj + 4 * grp]);
                const f32x4 ubj = *reinterpret_cast<const f32x4 *>(&sUb[c][16 * jj + 4 * grp]);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const f32x4 gv = gacc[d][mt];
                    f32x4 m;
                    if (jj < mt) {          // forward decay from j to t, all j < t
                        const float at = lat[mt] * ex2(Eb[mt - 1] - Eb[jj]);
#pragma unroll
                        for (int r = 0; r < 4; ++r) m[r] = gv[r] * at * lbj[r];
                    } else if (jj > mt) {   // reverse decay a_t ... a_{j-1}, all j > t
                        const float at = uat[mt] * ex2(Xb(jj) - Xb(mt + 1));
#pragma unroll
                        for (int r = 0; r < 4; ++r) m[r] = gv[r] * at * ubj[r];
                    } else {                // both, and the token's own input twice
                        const int t = 16 * mt + col;
                        const f32x4 csj = *reinterpret_cast<const f32x4 *>(&sCs[c][16 * jj + 4 * grp]);
                        const f32x4 exj = *reinterpret_cast<const f32x4 *>(&sEx[c][16 * jj + 4 * grp]);
                        const f32x4 dtj = *reinterpret_cast<const f32x4 *>(&sDt[c][16 * jj + 4 * grp]);
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int j = 16 * jj + 4 * grp + r;
                            const float e = ex2(j < t ? cst[mt] - csj[r] : exj[r] - ext[mt]);
                            m[r] = gv[r] * (j == t ? 2.f : e) * dtj[r];
                        }
                    }
                    s16x4 hh, ll;
                    split4(m, hh, ll);
                    mh[d][mt] = as_u2(hh);
                    ml[d][mt] = as_u2(ll);
                }
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const s16x4 x0 = as_s16x4(xq[jt]), x1 = as_s16x4(xq[jt + 1]);
                Y[mt] = mma_k32(as_s16x4(mh[0][mt]), as_s16x4(mh[1][mt]), x0, x1, Y[mt]);
                Y[mt] = mma_k32(as_s16x4(ml[0][mt]), as_s16x4(ml[1][mt]), x0, x1, Y[mt]);
            }
        }
    }

    // the cached state's slice (every wave: the forward state entering its chunk starts
    // from it)
    const int64_t slot = a.use_slots ? a.slots[b] : b;
    float *st = a.pool + (slot * a.nheads + h) * (kP * NS);
    f32x4 S[QN];
#pragma unroll
    for (int q = 0; q < QN; ++q) S[q] = *reinterpret_cast<const f32x4 *>(st + quad_off(q, grp, p));

    // ---- local states of the chunk (forward: needed by later chunks and by a commit;
    // reverse: by earlier chunks), contracted over tokens against B read transposed
    const bool need_f = COMMIT || c + 1 < NCH;
    const bool need_r = want_y && c > 0;
    f32x4 F[QN], R[QN];
    {
        Terms<COMMIT> wf[4];
        Terms<false> wr[4];
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            const f32x4 xv = bf16x4_val(xq[jt]);
            wf[jt] = terms<COMMIT>(*reinterpret_cast<const f32x4 *>(&sWf[c][16 * jt + 4 * grp]) * xv);
            wr[jt] = terms<false>(*reinterpret_cast<const f32x4 *>(&sWr[c][16 * jt + 4 * grp]) * xv);
        }
        // B read transposed: tokens 16jt + 4grp + r at dstate 16q + col, one dstate tile
        // ahead of the products that use it
        auto gather = [&](int q, uint32_t (&e)[16]) {
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
#pragma unroll
                for (int r = 0; r < 4; ++r) e[4 * jt + r] = img[(16 * jt + 4 * grp + r) * RS + 16 * q + col];
        };
        uint32_t eb[2][16];   // two buffers, alternating (indices fixed after unrolling)
        gather(0, eb[0]);
#pragma unroll
        for (int q = 0; q < QN; ++q) {
            if (q + 1 < QN) gather(q + 1, eb[(q + 1) & 1]);
            const uint32_t *ecur = eb[q & 1];
            uint2 bt[4];
#pragma unroll
            for (int jt = 0; jt < 4; ++jt)
                bt[jt] = uint2{ecur[4 * jt] | (ecur[4 * jt + 1] << 16), ecur[4 * jt + 2] | (ecur[4 * jt + 3] << 16)};
            F[q] = R[q] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (need_f) F[q] = mma_w<COMMIT>(bt, wf, F[q]);
            if (need_r) R[q] = mma_w<false>(bt, wr, R[q]);
        }
    }
    // publish them (the wave's own reads of its B image are issued before these writes
    // and LDS serves a wave's instructions in order)
    f32x4 *pub = reinterpret_cast<f32x4 *>(sReg[c]);
#pragma unroll
    for (int q = 0; q < QN; ++q) {
        if (need_f) pub[(4 * q + grp) * 16 + col] = F[q];
        if (need_r) pub[QN * 64 + (4 * q + grp) * 16 + col] = R[q];
    }
    // the cached state is in registers before any wave can write the committed one
#pragma unroll
    for (int q = 0; q < QN; ++q) asm volatile("" : "+v"(S[q]));
    __syncthreads();

    // ---- the forward state entering the chunk, S_c, from the cached state and the
    // earlier chunks' local states
    for (int k = 0; k < c; ++k) {
        const float keep = ex2(sTot[k]);
        const f32x4 *src = reinterpret_cast<const f32x4 *>(sReg[k]);
#pragma unroll
        for (int q = 0; q < QN; ++q) S[q] = S[q] * keep + src[(4 * q + grp) * 16 + col];
    }
    // ---- commit: the state after the block, 2^{tot} S_{NCH-1} + F_{NCH-1} (its own
    // local state, read back from where it was published)
    if constexpr (COMMIT) {
        if (c == NCH - 1) {
            const float keep = ex2(tot);
            const f32x4 *own = reinterpret_cast<const f32x4 *>(sReg[c]);
#pragma unroll
            for (int q = 0; q < QN; ++q)
                *reinterpret_cast<f32x4 *>(st + quad_off(q, grp, p)) =
                    S[q] * keep + own[(4 * q + grp) * 16 + col];
        }
    }
    if (!want_y) return;

    // ---- prefix terms C_t . S_c (forward) and C_t . E_c (reverse), each scaled per token
    // (2^{cs_t}, 2^{tot - ex_t}) and added to the intra-chunk terms
    auto prefix = [&](const f32x4 (&St)[QN], const float *scale) {
        f32x4 Yt[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) Yt[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < QN; q += 2) {
            if constexpr (QN == 1) {
                s16x4 sh, sl2;
                split4(St[0], sh, sl2);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const s16x4 cc = as_s16x4(cq[mt][0]);
                    Yt[mt] = mma_k16(cc, sh, Yt[mt]);
                    Yt[mt] = mma_k16(cc, sl2, Yt[mt]);
                }
            } else {   // two dstate quads per product
                s16x4 h0, l0, h1, l1;
                split4(St[q], h0, l0);
                split4(St[q + 1], h1, l1);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const s16x4 c0 = as_s16x4(cq[mt][q]), c1 = as_s16x4(cq[mt][q + 1]);
                    Yt[mt] = mma_k32(c0, c1, h0, h1, Yt[mt]);
                    Yt[mt] = mma_k32(c0, c1, l0, l1, Yt[mt]);
                }
            }
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            Y[mt] += *reinterpret_cast<const f32x4 *>(&scale[16 * mt + 4 * grp]) * Yt[mt];
        }
    };
    prefix(S, sEc[c]);
    if (c + 1 < NCH) {
        // the reverse state entering the chunk from its right, E_c, from the later chunks
        f32x4 E[QN];
#pragma unroll
        for (int q = 0; q < QN; ++q) E[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int k = NCH - 1; k > c; --k) {
            const float keep = ex2(sTot[k]);
            const f32x4 *src = reinterpret_cast<const f32x4 *>(sReg[k]) + QN * 64;
#pragma unroll
            for (int q = 0; q < QN; ++q) E[q] = E[q] * keep + src[(4 * q + grp) * 16 + col];
        }
        prefix(E, sEr[c]);
    }

    // ---- skip term and store (lane (col, grp): token 16mt + 4grp + r, column p); tokens
    // past the block get an out-of-range offset and their stores are dropped
    const float skip = a.D[h] + a.D_rev[h];
    const __amdgpu_buffer_rsrc_t rY =
        rsrc(a.y + ((static_cast<int64_t>(b) * a.L + t0) * a.nheads + h) * kP + p0);
    const uint32_t ytokB = static_cast<uint32_t>(a.nheads) * kP * 4;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
        const f32x4 xv = bf16x4_val(xq[mt]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * mt + 4 * grp + r;
            const uint32_t o = t < lim ? (4 * grp + r) * ytokB + 4 * col : kOOB;
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(Y[mt][r] + skip * xv[r]), rY, o,
                                                  16 * mt * ytokB, kNT);
        }
    }
}

template <int NS, int NCH>
hipError_t long_launch(const LongArgs &k, bool commit, unsigned grid, hipStream_t s) {
    if (commit)
        hipLaunchKernelGGL((bdlm_long_block_kernel<NS, NCH, true>), dim3(grid), dim3(64 * NCH), 0, s, k);
    else
        hipLaunchKernelGGL((bdlm_long_block_kernel<NS, NCH, false>), dim3(grid), dim3(64 * NCH), 0, s, k);
    return hipGetLastError();
}
template <int NS>
hipError_t long_nch(const LongArgs &k, int nch, bool commit, unsigned grid, hipStream_t s) {
    switch (nch) {
        case 2: return long_launch<NS, 2>(k, commit, grid, s);
        case 3: return long_launch<NS, 3>(k, commit, grid, s);
        case 4: return long_launch<NS, 4>(k, commit, grid, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool long_chunked_fits(const LaunchArgs &a) {
    return a.bf16 && a.L > 64 && a.L <= 4 * kCh && a.batch <= BDLM_MAX_SLOT_ROWS &&
           (a.dstate == 16 || a.dstate == 32 || a.dstate == 64 || a.dstate == 128);
}

int launch_block_long_shared(const LaunchArgs &a, bool commit, bool want_y, void *stream) {
    return long_chunked_fits(a) ? launch_long_chunked(a, commit, want_y, stream)
                                : launch_block_long(a, a, commit, want_y, stream);
}

int launch_long_chunked(const LaunchArgs &a, bool commit, bool want_y, void *stream) {
    if (a.batch == 0 || a.L == 0) return BDLM_OK;
    if (!long_chunked_fits(a)) return BDLM_E_SHAPE;
    if (!commit && !want_y) return BDLM_OK;
    LongArgs k;
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
    const int64_t grid = static_cast<int64_t>(a.batch) * a.nheads * kSlices;
    k.xcd_remap = grid % 8 == 0 ? 1 : 0;
    const int nch = (a.L + kCh - 1) / kCh;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const unsigned gr = static_cast<unsigned>(grid);
    hipError_t e;
    switch (a.dstate) {
        case 16: e = long_nch<16>(k, nch, commit, gr, s); break;
        case 32: e = long_nch<32>(k, nch, commit, gr, s); break;
        case 64: e = long_nch<64>(k, nch, commit, gr, s); break;
        default: e = long_nch<128>(k, nch, commit, gr, s); break;
    }
    return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

}  // namespace bdlm
