// bdlm_chain.hip -- gfx950 kernels that run the selective scan along a whole
// sequence in 64-token chunks, carrying the state in registers from chunk to
// chunk: the full-window bidirectional scan (forward over the window from zero
// plus reverse over the window from zero, Sec. 4 and Sec. 5.1: the full-sequence
// DiffuMamba-style scan the paper contrasts with its block-restricted one), and
// the chunked prefix prefill (a clean prefix summarised into the cached forward
// state, Eq. boundary-state).
//
// Per chunk [s, e) of the sequence, with l_t = dt_t A_h, local inclusive sums
// cs_t = l_s + ... + l_t, exclusive ex_t = cs_{t-1} (ex_s = 0), total = cs_{e-1}:
//   forward   y_t = exp(cs_t) (C_t . S_in) + sum_{j<=t} exp(cs_t - cs_j) (C_t.B_j) dt_j x_j
//                   + D x_t
//             S_out = exp(total) S_in + sum_j exp(total - cs_j) dt_j x_j (outer) B_j
//   reverse   y_t = exp(total - ex_t) (C_t . R_in) + sum_{j>=t} exp(ex_j - ex_t) (C_t.B_j) dt_j x_j
//                   + D_rev x_t
//             R_out = exp(total) R_in + sum_j exp(ex_j) dt_j x_j (outer) B_j
// where S_in is the forward state before the chunk (zero, or the cached state for
// a prefill) and R_in the reverse state after it (zero past the end).  The forward
// pass walks the chunks in order, the reverse pass backwards and adds its outputs
// into y.  Padding past the end of the sequence (dt = 0, x = B = C = 0) changes
// nothing.
//
// Work decomposition: the state rows p are independent, so a head is split over
// 64 / (16 PB) workgroups by head-dim columns; inside a workgroup, wave (pb, part)
// owns 16 columns and one share of the dstate quads.  Per chunk the workgroup
// stages B, C (as MFMA register images), its x columns and dt in LDS, builds the
// directional decay-weighted Gram matrix once, and every wave contracts it with
// x, contracts C with its state quads and updates them; the loads of the next
// chunk are in flight during the current chunk's arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_device.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

constexpr int kLC = 64;           // chunk length (tokens): one token per lane in the scans
constexpr int kMT = kLC / 16;     // token tiles per chunk

struct CArgs {
    const void *x, *dt, *Bm, *Cm;
    const float *A, *skip;        // skip: D (forward pass) or D_rev (reverse pass)
    float *h_pool;                // prefill: states read and written; else nullptr (zero start)
    float *y;                     // nullptr: no outputs
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int64_t T;                    // tokens in the sequence
    int32_t nheads, heads_per_group;
    int32_t accumulate;           // 1: y += this pass's outputs
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

// NS: dstate.  F32: fp32 activation storage.  REV: reverse pass.  NPART: dstate
// shares (wave groups).  PB: 16-column blocks per workgroup (64 / (16 PB)
// workgroups per head).
template <int NS, bool F32, bool REV, int NPART, int PB>
__global__ void __launch_bounds__(64 * PB * NPART)
bdlm_chain_kernel(const CArgs args) {
    constexpr int NT = 64 * PB * NPART;   // threads
    constexpr int NW = PB * NPART;        // waves
    constexpr int MT = kMT;
    constexpr int QN = NS / 16;
    constexpr int QW = QN / NPART;
    static_assert(QN % NPART == 0 && QW >= 1, "dstate split");
    constexpr int IMG = MT * QN * 64;
    constexpr int E = F32 ? 4 : 8;        // activations per 16-byte chunk
    constexpr int XCOLS = 16 * PB;        // head-dim columns of this workgroup
    constexpr int XS = XCOLS + 4;         // x row stride in LDS (elements)
    constexpr int WPH = 4 / PB;           // workgroups per head
    using AT = typename Act<F32>::T;

    __shared__ __align__(16) uint2 sC[IMG], sB[IMG];
    __shared__ __align__(16) uint2 sCl[F32 ? IMG : 1], sBl[F32 ? IMG : 1];
    __shared__ __align__(16) AT sX[kLC * XS];
    __shared__ __align__(16) float sDt[64];
    __shared__ __align__(16) uint4 sM[MT * MT * 64];
    __shared__ __align__(16) f32x4 sRed[(NPART > 1 ? NPART - 1 : 1) * PB * MT * 64];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int pb = wave % PB, part = wave / PB;
    const int col = lane & 15, grp = lane >> 4;

    const int u = blockIdx.x / WPH, wslice = blockIdx.x % WPH;
    const int b = u / args.nheads;
    const int h = u - b * args.nheads;
    const int g = h / args.heads_per_group;
    const int pc0 = wslice * XCOLS;          // first head-dim column of this workgroup
    const int p = pc0 + pb * 16 + col;       // this lane's column
    const int xc = pb * 16 + col;            // ... within the workgroup's x slice
    const int q0 = part * QW;
    const int64_t T = args.T;
    const int nch = static_cast<int>((T + kLC - 1) / kLC);

    const AT *xg = static_cast<const AT *>(args.x) + b * args.xs_b + h * args.xs_h + pc0;
    const AT *dtg = static_cast<const AT *>(args.dt) + b * args.dts_b + h;
    const AT *Bg = static_cast<const AT *>(args.Bm) + b * args.bcs_b + g * args.bcs_g;
    const AT *Cg = static_cast<const AT *>(args.Cm) + b * args.bcs_b + g * args.bcs_g;
    typedef __attribute__((address_space(1))) const AT g_at;

    const float A2 = args.A[h] * kLog2e;    // base 2 throughout
    const float skip = args.skip[h];

    // ---- the carried state: this lane's quads s[p, 16q + 4grp + r], q = q0 + k
    f32x4 st[QW];
    float *hs = nullptr;
    if (args.h_pool) {
        const int64_t slot = args.use_slots ? args.slots[b] : b;
        hs = args.h_pool + (slot * args.nheads + h) * kP * NS + (grp * kP + p) * 4;
#pragma unroll
        for (int k = 0; k < QW; ++k)
            st[k] = *reinterpret_cast<const f32x4 *>(hs + (q0 + k) * 16 * kP);
    } else {
#pragma unroll
        for (int k = 0; k < QW; ++k) st[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // ---- chunk loads into registers (issued one chunk ahead)
    constexpr int CPR = NS / E;
    constexpr int BC_CH = kLC * CPR;
    constexpr int BC_PT = BC_CH >= NT ? BC_CH / NT : 1;
    const bool bc_owner = tid < BC_CH;
    constexpr int X_CPR = XCOLS / E;
    constexpr int X_CH = kLC * X_CPR;
    constexpr int X_PT = X_CH >= NT ? X_CH / NT : 1;
    const bool x_owner = tid < X_CH;
    u32x4 cch[BC_PT], bch[BC_PT], xch[X_PT];
    AT dtraw = AT(0);
    auto issue = [&](int c) {
        const int64_t t0 = static_cast<int64_t>(c) * kLC;
        if (bc_owner) {
#pragma unroll
            for (int k = 0; k < BC_PT; ++k) {
                const int i = tid + NT * k;
                const int t = i / CPR, cc = i % CPR;
                const bool ok = t0 + t < T;
                const int64_t o = (t0 + t) * args.bcs_t + cc * E;
                cch[k] = *(ok ? gchunk(Cg + o) : gzero());
                bch[k] = *(ok ? gchunk(Bg + o) : gzero());
            }
        }
        if (x_owner) {
#pragma unroll
            for (int k = 0; k < X_PT; ++k) {
                const int i = tid + NT * k;
                const int j = i / X_CPR, cc = i % X_CPR;
                xch[k] = *(t0 + j < T ? gchunk(xg + (t0 + j) * args.xs_t + cc * E) : gzero());
            }
        }
        if (wave == 0)
            dtraw = *(t0 + lane < T ? (const g_at *)(dtg + (t0 + lane) * args.dts_t)
                                    : (const g_at *)(&kZeroChunk));
    };

    const uint16_t *sBh = reinterpret_cast<const uint16_t *>(sB);
    const uint16_t *sBlo = reinterpret_cast<const uint16_t *>(sBl);

    issue(REV ? nch - 1 : 0);
    for (int it = 0; it < nch; ++it) {
        const int c = REV ? nch - 1 - it : it;
        const int64_t t0 = static_cast<int64_t>(c) * kLC;
        const int valid = T - t0 < kLC ? static_cast<int>(T - t0) : kLC;

        // ---- stage this chunk in LDS, then start loading the next one
#pragma unroll
        for (int k = 0; k < BC_PT; ++k) {
            if (!bc_owner) break;
            const int i = tid + NT * k;
            const int t = i / CPR, cc = i % CPR;
            const u32x4 cz = cch[k], bz = bch[k];
            if constexpr (F32) {
                const int at = img_idx<QN, F32>(t >> 4, cc >> 2, cc & 3, t & 15);
                s16x4 hi, lo;
                split4(__builtin_bit_cast(f32x4, cz), hi, lo);
                sC[at] = as_u2(hi);
                sCl[at] = as_u2(lo);
                split4(__builtin_bit_cast(f32x4, bz), hi, lo);
                sB[at] = as_u2(hi);
                sBl[at] = as_u2(lo);
            } else {
                const int at = img_idx<QN, F32>(t >> 4, cc >> 1, 2 * (cc & 1), t & 15);
                sC[at] = uint2{cz.x, cz.y};
                sC[at + 16] = uint2{cz.z, cz.w};
                sB[at] = uint2{bz.x, bz.y};
                sB[at + 16] = uint2{bz.z, bz.w};
            }
        }
        if (x_owner) {
#pragma unroll
            for (int k = 0; k < X_PT; ++k) {
                const int i = tid + NT * k;
                const int j = i / X_CPR, cc = i % X_CPR;
                const u32x4 v = xch[k];
                uint2 *dst = reinterpret_cast<uint2 *>(&sX[j * XS + cc * E]);
                dst[0] = uint2{v.x, v.y};
                dst[1] = uint2{v.z, v.w};
            }
        }
        if (wave == 0) sDt[lane] = Act<F32>::val(dtraw);
        __syncthreads();
        // the outputs to add to (reverse pass), loaded before the next chunk's
        // prefetch so that waiting for them never waits for the prefetch
        float *yrow = nullptr;
        const int64_t ytok = static_cast<int64_t>(args.nheads) * kP;
        float yacc[MT][4];
        if (args.y && part == 0) {
            yrow = args.y + ((static_cast<int64_t>(b) * T + t0 + 4 * grp) * args.nheads + h) * kP + p;
            if (args.accumulate) {
                typedef __attribute__((address_space(1))) const float g_fl;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        yacc[mt][r] = *(16 * mt + 4 * grp + r < valid
                                            ? (const g_fl *)(yrow + (16 * mt + r) * ytok)
                                            : (const g_fl *)(&kZeroChunk));
            } else {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) yacc[mt][r] = 0.f;
            }
        }
        if (it + 1 < nch) issue(REV ? c - 1 : c + 1);

        // ---- decay prefix sums of the chunk (lane t = token t)
        const float dtv = sDt[lane];
        const float l2 = dtv * A2;
        float cs = l2;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const float v = __shfl_up(cs, off, 64);
            if (lane >= off) cs += v;
        }
        float ex = __shfl_up(cs, 1, 64);
        if (lane == 0) ex = 0.f;
        const float total = shfl(cs, 63);

        // ---- directional decay-weighted Gram tiles, shared out over the waves
        for (int tile = wave; tile < MT * MT; tile += NW) {
            const int mt = tile / MT, jt = tile % MT;
            const int t = 16 * mt + col;
            f32x4 m = {0.f, 0.f, 0.f, 0.f};
            // tiles entirely on the masked side stay zero
            const bool live = REV ? (jt >= mt) : (jt <= mt);
            if (live) {
                f32x4 gacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < QN; q += 2) {
                    const int q1 = q + 1 < QN ? q + 1 : q;
                    const s16x4 b0 = as_s16x4(sB[img_idx<QN, F32>(jt, q, grp, col)]);
                    const s16x4 b1 = as_s16x4(sB[img_idx<QN, F32>(jt, q1, grp, col)]);
                    const s16x4 c0 = as_s16x4(sC[img_idx<QN, F32>(mt, q, grp, col)]);
                    const s16x4 c1 = as_s16x4(sC[img_idx<QN, F32>(mt, q1, grp, col)]);
                    if (q + 1 < QN) gacc = mma_k32(b0, b1, c0, c1, gacc);
                    else gacc = mma_k16(b0, c0, gacc);
                    if constexpr (F32) {
                        const s16x4 bl0 = as_s16x4(sBl[img_idx<QN, F32>(jt, q, grp, col)]);
                        const s16x4 bl1 = as_s16x4(sBl[img_idx<QN, F32>(jt, q1, grp, col)]);
                        const s16x4 cl0 = as_s16x4(sCl[img_idx<QN, F32>(mt, q, grp, col)]);
                        const s16x4 cl1 = as_s16x4(sCl[img_idx<QN, F32>(mt, q1, grp, col)]);
                        if (q + 1 < QN) {
                            gacc = mma_k32(b0, b1, cl0, cl1, gacc);
                            gacc = mma_k32(bl0, bl1, c0, c1, gacc);
                        } else {
                            gacc = mma_k16(b0, cl0, gacc);
                            gacc = mma_k16(bl0, c0, gacc);
                        }
                    }
                }
                const float cst = shfl(cs, t), ext = shfl(ex, t);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    // shuffles outside the selects: a lane shuffle only sees the
                    // values of lanes that execute it
                    const int j = 16 * jt + 4 * grp + r;
                    const float dtj = shfl(dtv, j), csj = shfl(cs, j), exj = shfl(ex, j);
                    float w;
                    if constexpr (REV) w = j >= t ? exp2f(exj - ext) : 0.f;
                    else w = j <= t ? exp2f(cst - csj) : 0.f;
                    m[r] = gacc[r] * w * dtj;
                }
            }
            s16x4 mh, ml;
            split4(m, mh, ml);
            const uint2 a = as_u2(mh), c2 = as_u2(ml);
            sM[tile * 64 + lane] = uint4{a.x, a.y, c2.x, c2.y};
        }
        __syncthreads();

        // ---- x quads of this wave's columns (B operand, j = 16jt + 4grp + r)
        float xv[MT][4];
        s16x4 xq[MT], xl[MT];
#pragma unroll
        for (int jt = 0; jt < MT; ++jt) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                xv[jt][r] = Act<F32>::val(sX[(16 * jt + 4 * grp + r) * XS + xc]);
            split4(f32x4{xv[jt][0], xv[jt][1], xv[jt][2], xv[jt][3]}, xq[jt], xl[jt]);
        }

        if (args.y) {
            // partial products with this wave's state quads
            f32x4 ap[MT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                ap[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int k = 0; k < QW; k += 2) {
                    if (k + 1 < QW) {
                        s16x4 h0, l0, h1, l1;
                        split4(st[k], h0, l0);
                        split4(st[k + 1], h1, l1);
                        const s16x4 c0 = as_s16x4(sC[img_idx<QN, F32>(mt, q0 + k, grp, col)]);
                        const s16x4 c1 = as_s16x4(sC[img_idx<QN, F32>(mt, q0 + k + 1, grp, col)]);
                        ap[mt] = mma_k32(c0, c1, h0, h1, ap[mt]);
                        ap[mt] = mma_k32(c0, c1, l0, l1, ap[mt]);
                        if constexpr (F32) {
                            const s16x4 d0 = as_s16x4(sCl[img_idx<QN, F32>(mt, q0 + k, grp, col)]);
                            const s16x4 d1 =
                                as_s16x4(sCl[img_idx<QN, F32>(mt, q0 + k + 1, grp, col)]);
                            ap[mt] = mma_k32(d0, d1, h0, h1, ap[mt]);
                        }
                    } else {
                        s16x4 h0, l0;
                        split4(st[k], h0, l0);
                        const s16x4 c0 = as_s16x4(sC[img_idx<QN, F32>(mt, q0 + k, grp, col)]);
                        ap[mt] = mma_k16(c0, h0, ap[mt]);
                        ap[mt] = mma_k16(c0, l0, ap[mt]);
                        if constexpr (F32) {
                            const s16x4 d0 = as_s16x4(sCl[img_idx<QN, F32>(mt, q0 + k, grp, col)]);
                            ap[mt] = mma_k16(d0, h0, ap[mt]);
                        }
                    }
                }
            }
            if constexpr (NPART > 1) {
                if (part > 0)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        sRed[(((part - 1) * PB + pb) * MT + mt) * 64 + lane] = ap[mt];
                __syncthreads();
                if (part == 0)
#pragma unroll
                    for (int pt = 1; pt < NPART; ++pt)
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt)
                            ap[mt] += sRed[(((pt - 1) * PB + pb) * MT + mt) * 64 + lane];
            }
            if (part == 0) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    s16x4 mh[MT], ml[MT];
#pragma unroll
                    for (int jt = 0; jt < MT; ++jt) {
                        const uint4 v = sM[(mt * MT + jt) * 64 + lane];
                        mh[jt] = as_s16x4(uint2{v.x, v.y});
                        ml[jt] = as_s16x4(uint2{v.z, v.w});
                    }
                    f32x4 ai = {0.f, 0.f, 0.f, 0.f};
                    ai = mma_quads<MT>(mh, xq, ai);
                    ai = mma_quads<MT>(ml, xq, ai);
                    if constexpr (F32) ai = mma_quads<MT>(mh, xl, ai);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int t = 16 * mt + 4 * grp + r;
                        const float sc = REV ? exp2f(total - shfl(ex, t)) : exp2f(shfl(cs, t));
                        if (t < valid)
                            yrow[(16 * mt + r) * ytok] =
                                sc * ap[mt][r] + ai[r] + skip * xv[mt][r] + yacc[mt][r];
                    }
                }
            }
        }

        // ---- carry the state across the chunk
        {
            const float keep = exp2f(total);
            float wj[MT][4];
#pragma unroll
            for (int jt = 0; jt < MT; ++jt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int j = 16 * jt + 4 * grp + r;
                    const float e = REV ? exp2f(shfl(ex, j)) : exp2f(total - shfl(cs, j));
                    wj[jt][r] = e * shfl(dtv, j);
                }
#pragma unroll
            for (int k = 0; k < QW; ++k) {
                const int q = q0 + k;
                s16x4 th[MT], tl[MT];
#pragma unroll
                for (int jt = 0; jt < MT; ++jt) {
                    f32x4 v;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int e = img_idx<QN, F32>(jt, q, col >> 2, 4 * grp + r) * 4 + (col & 3);
                        float bv = bf16_to_f32(static_cast<short>(sBh[e]));
                        if constexpr (F32) bv += bf16_to_f32(static_cast<short>(sBlo[e]));
                        v[r] = bv * wj[jt][r];
                    }
                    split4(v, th[jt], tl[jt]);
                }
                f32x4 acc = st[k] * keep;
                acc = mma_quads<MT>(th, xq, acc);
                acc = mma_quads<MT>(tl, xq, acc);
                if constexpr (F32) acc = mma_quads<MT>(th, xl, acc);
                st[k] = acc;
            }
        }
        __syncthreads();   // LDS is rewritten by the next chunk
    }

    if (hs) {
#pragma unroll
        for (int k = 0; k < QW; ++k)
            *reinterpret_cast<f32x4 *>(hs + (q0 + k) * 16 * kP) = st[k];
    }
}

template <int NS, bool F32, bool REV>
hipError_t launch_chain_t(const CArgs &k, int units, hipStream_t s) {
    // two workgroups of 8 waves (2 column blocks x 2 dstate shares) per head when
    // dstate allows two shares, else four waves of one share
    constexpr int NP = (NS / 16) % 2 == 0 ? 2 : 1;
    constexpr int PB = 2;
    hipLaunchKernelGGL((bdlm_chain_kernel<NS, F32, REV, NP, PB>), dim3(units * (4 / PB)),
                       dim3(64 * PB * NP), 0, s, k);
    return hipGetLastError();
}

template <bool F32, bool REV>
hipError_t chain_by_ns(int ns, const CArgs &k, int units, hipStream_t s) {
    switch (ns) {
        case 16: return launch_chain_t<16, F32, REV>(k, units, s);
        case 32: return launch_chain_t<32, F32, REV>(k, units, s);
        case 64: return launch_chain_t<64, F32, REV>(k, units, s);
        case 128: return launch_chain_t<128, F32, REV>(k, units, s);
        default: return hipErrorInvalidValue;
    }
}

CArgs chain_args(const LaunchArgs &a, int64_t T) {
    CArgs k;
    k.x = a.x;
    k.dt = a.dt;
    k.Bm = a.Bm;
    k.Cm = a.Cm;
    k.A = a.A;
    k.skip = a.D;
    k.h_pool = nullptr;
    k.y = a.y;
    k.xs_b = a.xs_b;
    k.xs_t = a.xs_t;
    k.xs_h = a.xs_h;
    k.dts_b = a.dts_b;
    k.dts_t = a.dts_t;
    k.bcs_b = a.bcs_b;
    k.bcs_t = a.bcs_t;
    k.bcs_g = a.bcs_g;
    k.T = T;
    k.nheads = a.nheads;
    k.heads_per_group = a.nheads / a.ngroups;
    k.accumulate = 0;
    k.use_slots = a.slots ? 1 : 0;
    for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i)
        k.slots[i] = (a.slots && i < a.batch) ? a.slots[i] : 0;
    return k;
}

hipError_t run_chain(const CArgs &k, bool f32, bool rev, int ns, int units, hipStream_t s) {
    if (f32) return rev ? chain_by_ns<true, true>(ns, k, units, s) : chain_by_ns<true, false>(ns, k, units, s);
    return rev ? chain_by_ns<false, true>(ns, k, units, s) : chain_by_ns<false, false>(ns, k, units, s);
}

}  // namespace

int launch_full_window(const LaunchArgs &a, int64_t T, void *stream) {
    if (a.batch == 0 || T == 0) return BDLM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int units = a.batch * a.nheads;
    CArgs k = chain_args(a, T);
    k.use_slots = 0;
    k.skip = a.D;
    if (run_chain(k, !a.bf16, false, a.dstate, units, s) != hipSuccess) return BDLM_E_LAUNCH;
    k.skip = a.D_rev;
    k.accumulate = 1;
    if (run_chain(k, !a.bf16, true, a.dstate, units, s) != hipSuccess) return BDLM_E_LAUNCH;
    return BDLM_OK;
}

int launch_prefill(const LaunchArgs &a, int64_t T, void *stream) {
    if (a.batch == 0 || T == 0) return BDLM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    CArgs k = chain_args(a, T);
    k.h_pool = a.h_pool;
    k.skip = a.D;
    return run_chain(k, !a.bf16, false, a.dstate, a.batch * a.nheads, s) == hipSuccess
               ? BDLM_OK
               : BDLM_E_LAUNCH;
}

}  // namespace bdlm
