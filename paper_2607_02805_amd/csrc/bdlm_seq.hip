// bdlm_seq.hip -- gfx950 kernels that run the selective scan along whole sequences:
// the full-window bidirectional scan (forward over the window from a zero state plus
// reverse over it from a zero state, Sec. 4 and Sec. 5.1: the full-sequence scan the
// block-restricted one replaces) and the chunked prefill of a clean prefix into the
// cached forward states (Eq. boundary-state).
//
// The sequence is cut into segments of S tokens (a multiple of the 64-token chunk),
// and every (batch row, head, segment) is one workgroup:
//   seg_state    each segment's local states from zero -- forward F_k and, for the
//                full window, reverse R_k -- and its total log-decay T_k;
//   seg_combine  per state element, one pass over the segments turns these into the
//                states entering every segment:
//                  Sin_0 = s0,  Sin_{k+1} = 2^{T_k} Sin_k + F_k,
//                  Rin_{K-1} = 0,  Rin_{k-1} = 2^{T_k} Rin_k + R_k,
//                and for a prefill writes the final state 2^{T_{K-1}} Sin_{K-1} + F_{K-1}
//                back to the cache;
//   seg_out      the outputs of each segment in 64-token chunks from its entering state
//                (the reverse pass reads the forward pass's outputs a chunk at a time
//                and stores the sums: one reader and writer per element, no atomics).
// The reverse direction is the forward scan of the time-reversed sequence (every
// token keeps its own x, dt, B, C), so seg_out loads each chunk flipped and walks
// the segment's chunks backwards with the forward arithmetic.
//
// Per chunk, with l_i = dt_i A_h log2(e), inclusive sums cs_i and tot = cs_63:
//   y_i = 2^{cs_i} (C_i . S) + sum_{j<=i} 2^{cs_i - cs_j} dt_j (C_i . B_j) x_j + skip x_i
//   S  <- 2^{tot} S + sum_j 2^{tot - cs_j} dt_j x_j (outer) B_j
// Tokens outside the segment load as zeros (dt = 0: decay 1, no input), which
// changes nothing.
//
// Work split: 4 waves, wave w owns head-dim columns 16w .. 16w+15 of the state and
// of y.  A chunk is staged once in LDS: B, C and x as row images (MFMA operands over
// dstate; in bf16 storage B and x are also read transposed, as operands over tokens,
// with the LDS transpose read), dt and its decay sums.  The
// decay-weighted Gram tiles C.B^T (10 lower-triangle 16x16 tiles) are shared out
// over the waves and published in LDS; each wave then forms its columns' y and
// updates its state rows on MFMA: bf16 storage on bf16 MFMA (fp32 operands such as
// states and decay-weighted tiles split hi + lo, the bf16 activations exact), fp32
// storage on fp32 MFMA (every operand fp32, e.g. convolution outputs, which would lose
// accuracy in a two-term bf16 split).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bdlm.h"
#include "bdlm_device.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

constexpr int kC = 64;           // chunk length (tokens): one token per lane in the scan
constexpr int kThreads = 256;    // 4 waves
constexpr int kTiles = 10;       // lower-triangle 16x16 tiles of a 64x64 chunk

struct SeqArgs {
    const void *x, *dt, *Bm, *Cm;
    const float *A, *skip;       // skip: D (forward) or D_rev (reverse)
    float *y;                    // seg_out: outputs; nullptr: none
    float *ws;                   // segment states [unit][seg][dirs][64 * N] (pool layout)
    float *tot;                  // segment log2-decays [unit][seg]
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int64_t T, S;                // tokens in the sequence; tokens per segment
    int32_t nseg, dirs;
    int32_t nheads, heads_per_group;
    int32_t zero_init;           // seg_out: every segment starts from zero (ws unused)
    int32_t xcd_remap;           // grid % 8 == 0: keep a (row, segment)'s heads on one XCD
    int32_t blk_major;           // states of (row, head, segment) at slot (row * nseg + segment)
                                 // * nheads + head (a pool of per-block states); else
                                 // (row * nheads + head) * nseg + segment
    // seg_out with one segment per row (a block step or commit of any length):
    const float *pool_in;        // the entering state from the cache (slot per row)
    float *pool_out;             // the final state written back to the cache (in place)
    // seg_out, forward: chunks of cstride (<= 64) tokens, and the state entering every
    // chunk written to emit[(row * emit_blocks + block) * nheads + head] (block = the
    // chunk's index in the sequence; segments hold whole chunks)
    int32_t cstride;
    float *emit;
    int64_t emit_blocks;
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

// Slot of workgroup (row, head, segment)'s states in ws (times dirs states each).
__device__ __forceinline__ int64_t state_slot(const SeqArgs &a, int b, int h, int seg) {
    return a.blk_major ? (static_cast<int64_t>(b) * a.nseg + seg) * a.nheads + h
                       : (static_cast<int64_t>(b) * a.nheads + h) * a.nseg + seg;
}

template <int NS, bool F32>
struct Geo {
    static constexpr int QN = NS / 16;               // dstate tiles
    static constexpr int E = F32 ? 4 : 8;            // activations per 16-byte load
    static constexpr int BCPR = NS / E;              // 16-byte pieces per B / C row
    static constexpr int BT = 16 * BCPR;             // (token quad, piece) tasks
    static constexpr int BPT = BT > kThreads ? BT / kThreads : 1;
    static constexpr int XCPR = kP / E;
    static constexpr int XROWS = F32 ? 4 : 2;        // token rows per x task
    static constexpr int XT = (kC / XROWS) * XCPR;
    static constexpr int XPT = XT > kThreads ? XT / kThreads : 1;
    static constexpr int IMG = 4 * QN * 64;          // quads of a row image
    static_assert(BT % kThreads == 0 || BT < kThreads, "B tasks");
    static_assert(XT % kThreads == 0 || XT < kThreads, "x tasks");
};

// x in LDS: a bf16 row image (quads of four columns), or fp32 quads of four tokens'
// values per (token quad g, column p).
template <bool F32> struct XQuad;
template <> struct XQuad<false> { using T = uint2; };
template <> struct XQuad<true> { using T = f32x4; };

__device__ __forceinline__ float ex2(float v) { return __builtin_amdgcn_exp2f(v); }

// c += a b over one quad on fp32 MFMA: instruction r contracts lane group g's value
// r, i.e. index 4g + r of the quad layout.
__device__ __forceinline__ f32x4 mma_f32q(f32x4 a, f32x4 b, f32x4 c) {
#pragma unroll
    for (int r = 0; r < 4; ++r) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r], b[r], c, 0, 0, 0);
    return c;
}
// The LDS operand images hold bf16 quads (uint2) for bf16 storage and fp32 quads
// (f32x4, in the same arrays at twice the size) for fp32 storage.
__device__ __forceinline__ f32x4 f32q(const uint2 *img, int i) {
    return reinterpret_cast<const f32x4 *>(img)[i];
}

// Decode the workgroup into (batch row, segment, head): consecutive units of one
// (row, segment) share B and C, so they are kept on one XCD.
struct Unit {
    int b, seg, h;
};
__device__ __forceinline__ Unit decode(const SeqArgs &a) {
    int u = blockIdx.x;
    if (a.xcd_remap) u = (u & 7) * (static_cast<int>(gridDim.x) >> 3) + (u >> 3);
    Unit r;
    r.h = u % a.nheads;
    const int rest = u / a.nheads;
    r.seg = rest % a.nseg;
    r.b = rest / a.nseg;
    return r;
}

// Buffer resources: chunks are addressed from a per-chunk base (uniform, in scalar
// registers) plus a fixed per-thread byte offset.  Rows outside the segment lie past the
// resource's range (forward: the resource ends after the chunk's valid rows; reverse:
// they get an out-of-range offset): their loads return zeros and their stores are
// dropped, with no branch.
constexpr uint32_t kOOB = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             0x7fffffff, 0x00020000);
}
// The same over the first `bytes` bytes only: an access whose per-lane offset lies past
// them loads zeros and a store there is dropped (the range check of a buffer resource with
// stride 0 covers the per-lane and immediate offsets, not the scalar offset, so accesses
// through such a resource pass their whole offset per lane).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_n(const void *base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             bytes, 0x00020000);
}
constexpr int kNT = 2;   // buffer cache policy: nontemporal

// Row images of B and C in bf16 storage: quad (local token t, dstate quad Q = n / 4) at
// row_slot<QN>(t, Q).  Blocks of 64 quads per (16-token tile, 16-wide dstate tile); in a
// block, quad a = Q % 4 of the tile fills a row of 16 slots, the token within the tile
// XOR-permuted with 4a and the dstate tile.  Three access patterns each touch 16 distinct
// 8-byte bank pairs per 16 lanes for dstate 64 and 128 (checked on the CPU): the staging
// writes (one token, 16 consecutive 16-byte pieces of its row), the operand reads over
// dstate (16 tokens, one quad) and the transposed reads (4 tokens x 4 quads).
template <int QN>
__device__ __forceinline__ int row_slot(int t, int Q) {
    const int q = Q >> 2, a = Q & 3;
    return ((t >> 4) * QN + q) * 64 + a * 16 + ((t & 15) ^ (4 * a) ^ (q & 7));
}
// Row image of x in bf16 storage: quad (local token t, column quad PQ = p / 4) at
// x_slot(t, PQ), the same scheme over column tiles w = PQ / 4 (16 columns, one wave's).
__device__ __forceinline__ int x_slot(int t, int PQ) {
    const int w = PQ >> 2, a = PQ & 3;
    return ((t >> 4) * 4 + w) * 64 + a * 16 + ((t & 15) ^ (4 * a) ^ ((w & 1) | ((w & 2) << 1)));
}
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
// LDS transpose read (gfx950): every lane reads four bf16 at its own 8-byte-aligned
// address, and within each group of 16 lanes, lane 4a + b receives element b of the words
// read by lanes a, a + 4, a + 8 and a + 12 of its group, in that order.  So when lane s
// of group kg reads the quad (token 4kg + s / 4, columns c0 + 4 (s % 4) .. +3) of a
// token-major image, lane (kg, col) receives column c0 + col of tokens 4kg .. 4kg + 3:
// the operand over tokens of an MFMA that contracts along the chunk.
__device__ __forceinline__ s16x4 ds_read_tr(const uint2 *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(const_cast<uint2 *>(p)));
}
// The quad lane `lane` reads for the transposed operand of 16-token tile jt: token
// 16jt + tr_tok(lane), column quad 4 c + tr_quad(lane) of column tile c.
__device__ __forceinline__ int tr_tok(int lane) { return 4 * (lane >> 4) + ((lane & 15) >> 2); }
__device__ __forceinline__ int tr_quad(int lane) { return lane & 3; }

// One chunk's global loads into registers and their staging into LDS.  Local token
// i of chunk c is the segment's token 64c + i (reverse: its 64c + i-th token from
// the end); row(i) is its position in the chunk's memory window.  bf16 storage stages
// row images only (B, C when loaded, x), read transposed where the contraction runs
// over tokens; fp32 storage stages row images of B and C and transposed images of B
// and x (quads of four tokens' fp32 values).
template <int NS, bool F32, bool REV, bool LOADC>
struct Stager {
    using G = Geo<NS, F32>;
    static constexpr int ES = F32 ? 4 : 2;

    const char *xg, *dtg, *Bg, *Cg;  // this (row, head / group) at token 0
    int64_t xrow, dtrow, bcrow;      // bytes between consecutive tokens
    int64_t s0, s1;
    int cstride;                     // tokens per chunk (64; forward: any <= 64)
    uint32_t ob[G::BPT][4], ox[G::XPT][G::XROWS], odt;   // per-thread byte offsets
    u32x4 rb[G::BPT][4], rc[LOADC ? G::BPT : 1][4], rx[G::XPT][G::XROWS];
    uint32_t dtraw;

    static constexpr bool kRev = REV;
    __device__ __forceinline__ static int row(int i) { return REV ? kC - 1 - i : i; }

    // first token of chunk c's memory window, and the number of valid local tokens
    __device__ __forceinline__ int64_t window(int c) const {
        return REV ? s1 - static_cast<int64_t>(kC) * (c + 1) : s0 + static_cast<int64_t>(cstride) * c;
    }
    __device__ __forceinline__ int valid(int c) const {
        const int64_t v = (s1 - s0) - static_cast<int64_t>(cstride) * c;
        return v < cstride ? static_cast<int>(v) : cstride;
    }
    __device__ __forceinline__ int nchunks() const {
        return static_cast<int>((s1 - s0 + cstride - 1) / cstride);
    }
    // global token of local token i of chunk c; false outside the segment
    __device__ __forceinline__ bool token(int c, int i, int64_t &t) const {
        t = window(c) + row(i);
        return i < valid(c);
    }

    __device__ __forceinline__ void init(int tid, int lane) {
#pragma unroll
        for (int k = 0; k < G::BPT; ++k) {
            const int task = tid + kThreads * k, g = task / G::BCPR, pc = task % G::BCPR;
#pragma unroll
            for (int r = 0; r < 4; ++r)
                ob[k][r] = static_cast<uint32_t>(row(4 * g + r) * bcrow + pc * 16);
        }
#pragma unroll
        for (int k = 0; k < G::XPT; ++k) {
            const int task = tid + kThreads * k, g = task / G::XCPR, pc = task % G::XCPR;
#pragma unroll
            for (int r = 0; r < G::XROWS; ++r)
                ox[k][r] = static_cast<uint32_t>(row(G::XROWS * g + r) * xrow + pc * 16);
        }
        odt = static_cast<uint32_t>(row(lane) * dtrow);
    }

    __device__ __forceinline__ void issue(int c, int tid, int wave, int lane) {
        const int64_t w = window(c);
        const int lim = valid(c);
        // Forward, the chunk's rows past the segment are its last ones: the resources end
        // after the valid rows, so those rows load as zeros with no per-row test.  In
        // reverse they are the first rows of the window and get an out-of-range offset.
        const __amdgpu_buffer_rsrc_t rB =
            REV ? rsrc(Bg + w * bcrow) : rsrc_n(Bg + w * bcrow, static_cast<int>(lim * bcrow));
        const __amdgpu_buffer_rsrc_t rC =
            REV ? rsrc(Cg + w * bcrow) : rsrc_n(Cg + w * bcrow, static_cast<int>(lim * bcrow));
        const __amdgpu_buffer_rsrc_t rX =
            REV ? rsrc(xg + w * xrow) : rsrc_n(xg + w * xrow, static_cast<int>(lim * xrow));
#pragma unroll
        for (int k = 0; k < G::BPT; ++k) {
            const int task = tid + kThreads * k;
            if (task < G::BT) {
                const int g = task / G::BCPR;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const uint32_t o = !REV || 4 * g + r < lim ? ob[k][r] : kOOB;
                    rb[k][r] = __builtin_amdgcn_raw_buffer_load_b128(rB, o, 0, 0);
                    if constexpr (LOADC) rc[k][r] = __builtin_amdgcn_raw_buffer_load_b128(rC, o, 0, 0);
                }
            }
        }
#pragma unroll
        for (int k = 0; k < G::XPT; ++k) {
            const int task = tid + kThreads * k;
            if (task < G::XT) {
                const int g = task / G::XCPR;
#pragma unroll
                for (int r = 0; r < G::XROWS; ++r) {
                    const uint32_t o = !REV || G::XROWS * g + r < lim ? ox[k][r] : kOOB;
                    rx[k][r] = __builtin_amdgcn_raw_buffer_load_b128(rX, o, 0, 0);
                }
            }
        }
        if (wave == 0) {
            const __amdgpu_buffer_rsrc_t rD =
                REV ? rsrc(dtg + w * dtrow) : rsrc_n(dtg + w * dtrow, static_cast<int>(lim * dtrow));
            const uint32_t o = !REV || lane < lim ? odt : kOOB;
            if constexpr (F32) dtraw = __builtin_amdgcn_raw_buffer_load_b32(rD, o, 0, 0);
            else dtraw = __builtin_amdgcn_raw_buffer_load_b16(rD, o, 0, 0);
        }
    }

    __device__ __forceinline__ float dt_value() const {
        return F32 ? __uint_as_float(dtraw) : __uint_as_float(dtraw << 16);
    }

    // Row image of B or C (operand over dstate) from one task's four token rows.
    __device__ __forceinline__ static void row_image(const u32x4 (&v)[4], int g, int pc,
                                                     uint2 *hi) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int j = 4 * g + r;
            if constexpr (F32) {
                const int at = img_idx<G::QN, true>(j >> 4, pc >> 2, pc & 3, j & 15);
                reinterpret_cast<f32x4 *>(hi)[at] = __builtin_bit_cast(f32x4, v[r]);
            } else {
                hi[row_slot<G::QN>(j, 2 * pc)] = uint2{v[r].x, v[r].y};
                hi[row_slot<G::QN>(j, 2 * pc + 1)] = uint2{v[r].z, v[r].w};
            }
        }
    }

    // Write the registers of the current chunk into LDS.  sb, sc: row images of B and
    // C (B always for bf16 storage, both only when C is loaded for fp32); bt: the
    // transposed B image (fp32 only); xt: x, a row image (bf16) or transposed (fp32).
    __device__ __forceinline__ void stage(int tid, uint2 *sb, uint2 *sc, uint2 *bt,
                                          typename XQuad<F32>::T *xt) const {
#pragma unroll
        for (int k = 0; k < G::BPT; ++k) {
            const int task = tid + kThreads * k;
            if (task < G::BT) {
                const int g = task / G::BCPR, pc = task % G::BCPR;
                if constexpr (LOADC || !F32) row_image(rb[k], g, pc, sb);
                if constexpr (LOADC) row_image(rc[k], g, pc, sc);
                if constexpr (F32) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        reinterpret_cast<f32x4 *>(bt)[g * NS + pc * 4 + e] =
                            f32x4{__uint_as_float(rb[k][0][e]), __uint_as_float(rb[k][1][e]),
                                  __uint_as_float(rb[k][2][e]), __uint_as_float(rb[k][3][e])};
                }
            }
        }
#pragma unroll
        for (int k = 0; k < G::XPT; ++k) {
            const int task = tid + kThreads * k;
            if (task < G::XT) {
                const int g = task / G::XCPR, pc = task % G::XCPR;
                if constexpr (F32) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        xt[g * kP + pc * 4 + e] =
                            f32x4{__uint_as_float(rx[k][0][e]), __uint_as_float(rx[k][1][e]),
                                  __uint_as_float(rx[k][2][e]), __uint_as_float(rx[k][3][e])};
                } else {
#pragma unroll
                    for (int r = 0; r < G::XROWS; ++r) {
                        const int t = G::XROWS * g + r;
                        xt[x_slot(t, 2 * pc)] = uint2{rx[k][r].x, rx[k][r].y};
                        xt[x_slot(t, 2 * pc + 1)] = uint2{rx[k][r].z, rx[k][r].w};
                    }
                }
            }
        }
    }
};

// Wave 0: the chunk's decay sums.  sDt = dt, sCs = cs (inclusive, base 2),
// sEc = 2^cs, sWs = 2^(tot - cs) dt, sWr = 2^(cs - l) dt (weights of the local
// reverse state, relative to the chunk start).
template <bool WITH_WR>
__device__ __forceinline__ void decay_sums(float dtv, float A2, int lane, float *sDt, float *sCs,
                                           float *sEc, float *sWs, float *sWr) {
    const float l2 = dtv * A2;
    const float cs = wave_inclusive_sum(l2);
    const float tot = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cs), 63));
    sDt[lane] = dtv;
    sCs[lane] = cs;
    sEc[lane] = ex2(cs);
    sWs[lane] = ex2(tot - cs) * dtv;
    if constexpr (WITH_WR) sWr[lane] = ex2(cs - l2) * dtv;
}

// Operand quad of x for lane (grp, col) of wave w: tokens 16jt + 4grp .. +3 of column
// p = 16w + col, as bf16 (bf16 storage, read transposed from the row image) and as fp32.
template <bool F32>
__device__ __forceinline__ void x_operand(const typename XQuad<F32>::T *xt, int jt, int wave,
                                          int lane, s16x4 &hi, f32x4 &val) {
    if constexpr (F32) {
        val = xt[(4 * jt + (lane >> 4)) * kP + 16 * wave + (lane & 15)];
        hi = s16x4{0, 0, 0, 0};
    } else {
        hi = ds_read_tr(xt + x_slot(16 * jt + tr_tok(lane), 4 * wave + tr_quad(lane)));
        val = f32x4{bf16_to_f32(hi[0]), bf16_to_f32(hi[1]), bf16_to_f32(hi[2]), bf16_to_f32(hi[3])};
    }
}

// The transposed-B operand quads of dstate tile q (tokens 16jt + 4grp .. +3,
// column 16q + col) and the state update of one 16 x 16 (dstate, column) tile over
// the chunk's 64 tokens: acc += B^T (wh + wl), wh + wl the weighted x quads.
template <bool F32> struct BtOps;
template <> struct BtOps<false> { s16x4 h[4]; };
template <> struct BtOps<true> { f32x4 f[4]; };
// weighted x quads: bf16 hi + lo, or hi + mid + lo when T3 (bf16 storage), or fp32 (fp32
// storage).  T3 is used where the updated state leaves the kernels (a cache, the states
// entering blocks): carried over many blocks, a two-term split's 2^-18 residual per
// input adds up to more than the parity bar allows on states near zero.
template <bool F32, bool T3 = false> struct WOps;
template <bool T3> struct WOps<false, T3> { s16x4 h[4], l[4], m[T3 ? 4 : 1]; };
template <bool T3> struct WOps<true, T3> { f32x4 f[4]; };
template <bool F32, bool T3>
__device__ __forceinline__ void w_set(WOps<F32, T3> &o, int jt, f32x4 v) {
    if constexpr (F32) o.f[jt] = v;
    else if constexpr (T3) split4x3(v, o.h[jt], o.m[jt], o.l[jt]);
    else split4(v, o.h[jt], o.l[jt]);
}
// bt: the B row image (bf16, read transposed) or the transposed fp32 B image.
template <int NS, bool F32>
__device__ __forceinline__ void bt_read(BtOps<F32> &o, const uint2 *bt, int q, int lane) {
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        if constexpr (F32) o.f[jt] = f32q(bt, (4 * jt + (lane >> 4)) * NS + 16 * q + (lane & 15));
        else o.h[jt] = ds_read_tr(bt + row_slot<NS / 16>(16 * jt + tr_tok(lane), 4 * q + tr_quad(lane)));
    }
}
template <bool F32, bool T3>
__device__ __forceinline__ f32x4 bt_mma(const BtOps<F32> &o, const WOps<F32, T3> &w, f32x4 acc) {
    if constexpr (F32) {
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) acc = mma_f32q(o.f[jt], w.f[jt], acc);
    } else {
#pragma unroll
        for (int jt = 0; jt < 4; jt += 2) {
            acc = mma_k32(o.h[jt], o.h[jt + 1], w.h[jt], w.h[jt + 1], acc);
            acc = mma_k32(o.h[jt], o.h[jt + 1], w.l[jt], w.l[jt + 1], acc);
            if constexpr (T3) acc = mma_k32(o.h[jt], o.h[jt + 1], w.m[jt], w.m[jt + 1], acc);
        }
    }
    return acc;
}

// State quads of this lane in the pool layout: s[p][16q + 4grp .. +3] at
// ((4q + grp) * 64 + p) * 4.
__device__ __forceinline__ int quad_off(int q, int grp, int p) { return ((4 * q + grp) * kP + p) * 4; }

// Point a stager at workgroup (row, head, segment)'s inputs.
template <class ST>
__device__ __forceinline__ void setup(ST &st, const SeqArgs &a, const Unit &un, int g, int tid,
                                      int lane) {
    constexpr int ES = ST::ES;
    st.xg = static_cast<const char *>(a.x) + (un.b * a.xs_b + un.h * a.xs_h) * ES;
    st.dtg = static_cast<const char *>(a.dt) + (un.b * a.dts_b + un.h) * ES;
    st.Bg = static_cast<const char *>(a.Bm) + (un.b * a.bcs_b + g * a.bcs_g) * ES;
    st.Cg = a.Cm ? static_cast<const char *>(a.Cm) + (un.b * a.bcs_b + g * a.bcs_g) * ES : nullptr;
    st.xrow = a.xs_t * ES;
    st.dtrow = a.dts_t * ES;
    st.bcrow = a.bcs_t * ES;
    st.s0 = static_cast<int64_t>(un.seg) * a.S;
    st.s1 = st.s0 + a.S < a.T ? st.s0 + a.S : a.T;
    st.cstride = ST::kRev ? kC : a.cstride;
    st.init(tid, lane);
}

// ------------------------------------------------------------------ seg_state
// Local forward state F (and, BOTH, reverse state R) of one segment from zero, and
// the segment's total log2-decay.
template <int NS, bool F32, bool BOTH>
__global__ void __launch_bounds__(kThreads, F32 ? 1 : 2) bdlm_seg_state_kernel(const SeqArgs a) {
    using G = Geo<NS, F32>;
    constexpr int QN = G::QN;
    // B: bf16 row image (read transposed) or fp32 transposed image; x likewise
    __shared__ __align__(16) uint2 sBt[F32 ? 2 * 16 * NS : G::IMG];
    __shared__ __align__(16) typename XQuad<F32>::T sXt[16 * kP];
    __shared__ __align__(16) float sDt[kC], sCs[kC], sEc[kC], sWs[kC], sWr[kC];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int p = 16 * wave + col;
    const Unit un = decode(a);
    const int g = un.h / a.heads_per_group;

    Stager<NS, F32, false, false> st;
    setup(st, a, un, g, tid, lane);
    const int nch = st.nchunks();
    const float A2 = a.A[un.h] * kLog2e;

    f32x4 F[QN], R[BOTH ? QN : 1];
#pragma unroll
    for (int q = 0; q < QN; ++q) {
        F[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (BOTH) R[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float off = 0.f;   // log2-decay of the segment's tokens before the current chunk
    // forward-only segment states become cached or emitted states: three-term splits
    constexpr bool T3 = !BOTH;

    st.issue(0, tid, wave, lane);
    for (int c = 0; c < nch; ++c) {
        st.stage(tid, sBt, nullptr, sBt, sXt);
        if (wave == 0)
            decay_sums<BOTH>(st.dt_value(), A2, lane, sDt, sCs, sEc, sWs, sWr);
        __syncthreads();
        if (c + 1 < nch) st.issue(c + 1, tid, wave, lane);

        const float tot = sCs[kC - 1];
        WOps<F32, T3> wf, wr;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            s16x4 xh;
            f32x4 xv;
            x_operand<F32>(sXt, jt, wave, lane, xh, xv);
            w_set(wf, jt, *reinterpret_cast<const f32x4 *>(&sWs[16 * jt + 4 * grp]) * xv);
            if constexpr (BOTH)
                w_set(wr, jt,
                           *reinterpret_cast<const f32x4 *>(&sWr[16 * jt + 4 * grp]) * xv * ex2(off));
        }
        const float keep = ex2(tot);
        BtOps<F32> cur, nxt;
        bt_read<NS, F32>(cur, sBt, 0, lane);
#pragma unroll
        for (int q = 0; q < QN; ++q) {
            if (q + 1 < QN) bt_read<NS, F32>(nxt, sBt, q + 1, lane);
            F[q] = bt_mma(cur, wf, F[q] * keep);
            if constexpr (BOTH) R[q] = bt_mma(cur, wr, R[q]);
            if (q + 1 < QN) cur = nxt;
            __builtin_amdgcn_sched_barrier(0);
        }
        off += tot;
        __syncthreads();   // LDS is rewritten by the next chunk
    }

    float *out = a.ws + state_slot(a, un.b, un.h, un.seg) * a.dirs * (kP * NS);
#pragma unroll
    for (int q = 0; q < QN; ++q) {
        *reinterpret_cast<f32x4 *>(out + quad_off(q, grp, p)) = F[q];
        if constexpr (BOTH) *reinterpret_cast<f32x4 *>(out + kP * NS + quad_off(q, grp, p)) = R[q];
    }
    if (tid == 0) a.tot[(static_cast<int64_t>(un.b) * a.nheads + un.h) * a.nseg + un.seg] = off;
}

// ------------------------------------------------------------------ seg_out
// SUB > 0 (forward, with an emission pool): 64-token chunks holding blocks of SUB (16
// or 32) tokens; the state is carried block by block and the state entering every
// block is written.  SUB == 0: one emitted block per chunk of cstride tokens.
// T3PAR: the carried state is written out (a cache commit or emitted block states), so
// its updates use three-term splits (always for SUB > 0).
template <int NS, bool F32, bool REV, int SUB, bool T3PAR = false>
__global__ void __launch_bounds__(kThreads, F32 ? 1 : 2) bdlm_seg_out_kernel(const SeqArgs a) {
    static_assert(SUB == 0 || (!REV && (SUB == 16 || SUB == 32)), "block length");
    static_assert(!(REV && T3PAR), "the reverse pass keeps no state");
    constexpr bool T3 = T3PAR || SUB > 0;
    using G = Geo<NS, F32>;
    constexpr int QN = G::QN;
    constexpr int IMG = G::IMG;
    __shared__ __align__(16) uint2 sB[(F32 ? 2 : 1) * IMG], sC[(F32 ? 2 : 1) * IMG];
    __shared__ __align__(16) uint2 sBt[F32 ? 2 * 16 * NS : 1];   // fp32: transposed B
    __shared__ __align__(16) typename XQuad<F32>::T sXt[16 * kP];
    __shared__ __align__(16) uint4 sM[kTiles * 64];
    __shared__ __align__(16) float sDt[kC], sCs[kC], sEc[kC], sWs[kC];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 15, grp = lane >> 4;
    const int p = 16 * wave + col;
    const Unit un = decode(a);
    const int g = un.h / a.heads_per_group;

    Stager<NS, F32, REV, true> st;
    setup(st, a, un, g, tid, lane);
    const int nch = st.nchunks();
    const float A2 = a.A[un.h] * kLog2e;
    const float skip = a.skip[un.h];

    // the state entering the segment (in this direction's scan order)
    f32x4 S[QN];
    const int64_t cslot = a.use_slots ? a.slots[un.b] : un.b;
    if (a.pool_in) {
        const float *src = a.pool_in + (cslot * a.nheads + un.h) * (kP * NS);
#pragma unroll
        for (int q = 0; q < QN; ++q) S[q] = *reinterpret_cast<const f32x4 *>(src + quad_off(q, grp, p));
    } else if (a.zero_init) {
#pragma unroll
        for (int q = 0; q < QN; ++q) S[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    } else {
        const float *src =
            a.ws + (state_slot(a, un.b, un.h, un.seg) * a.dirs + (REV ? 1 : 0)) * (kP * NS);
#pragma unroll
        for (int q = 0; q < QN; ++q) S[q] = *reinterpret_cast<const f32x4 *>(src + quad_off(q, grp, p));
    }
    // The state loads complete here, before the chunk loop.  Otherwise the compiler's wait
    // analysis carries the pending loads into the loop: the first use of each quad in
    // every chunk then waits on the vector-memory counter, which from the second chunk on
    // means waiting for the next chunk's prefetched inputs (their full latency, every
    // chunk).
#pragma unroll
    for (int q = 0; q < QN; ++q) asm volatile("" : "+v"(S[q]));
    // states entering the segment's chunks (blocks), forward only
    float *emit_base = nullptr;
    int64_t emit_first = 0;
    if (!REV && a.emit) {
        emit_first = (static_cast<int64_t>(un.seg) * a.S) / (SUB > 0 ? SUB : a.cstride);
        emit_base = a.emit + (static_cast<int64_t>(un.b) * a.emit_blocks * a.nheads + un.h) * (kP * NS);
        float *dst = emit_base + emit_first * a.nheads * (kP * NS);
#pragma unroll
        for (int q = 0; q < QN; ++q) *reinterpret_cast<f32x4 *>(dst + quad_off(q, grp, p)) = S[q];
    }

    // y of this (row, head) at token 0, bytes between tokens, and this lane's offset of
    // local token 4grp within a chunk's memory window (tokens 16mt + r further on)
    const float *ybase = a.y + (static_cast<int64_t>(un.b) * a.T * a.nheads + un.h) * kP;
    const int64_t ytokB = static_cast<int64_t>(a.nheads) * kP * 4;
    const uint32_t oy = static_cast<uint32_t>(Stager<NS, F32, REV, true>::row(4 * grp) * ytokB + p * 4);
    // Full chunks (every local token inside the segment) address y as this lane's fixed
    // offset oyf plus a wave-uniform offset per (mt, r) in a scalar register, with no
    // per-access range test: local token 4grp + i sits at oyf + ysoff(i).  Partial chunks
    // keep a tested per-lane offset: the buffer range check does not see scalar offsets.
    const uint32_t oyf = REV ? oy - static_cast<uint32_t>(51 * ytokB) : oy;
    auto ysoff = [&](int i) { return static_cast<int>((REV ? 51 - i : i) * ytokB); };

    st.issue(0, tid, wave, lane);
    for (int c = 0; c < nch; ++c) {
        st.stage(tid, sB, sC, sBt, sXt);
        if (wave == 0)
            decay_sums<false>(st.dt_value(), A2, lane, sDt, sCs, sEc, sWs, nullptr);
        __syncthreads();
        // the next chunk's loads (the reverse pass, which also holds the y values it adds
        // onto, requests them after the Gram tiles instead: fewer registers live across the
        // Gram and prefix phase)
        if (!REV && c + 1 < nch) st.issue(c + 1, tid, wave, lane);
        // the reverse pass adds onto the forward pass's outputs: this lane's 16 of them are
        // requested now, before the chunk's products, and stored back with the sums (one
        // reader and writer per element, so the sum is exact fp32 and deterministic)
        float yv[REV ? 16 : 1];
        if constexpr (REV) {
            if (a.y) {
                const __amdgpu_buffer_rsrc_t rYl = rsrc(ybase + st.window(c) * (ytokB / 4));
                const int lim = st.valid(c);
                if (lim == kC) {
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        yv[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                            rYl, oyf, ysoff(16 * (i >> 2) + (i & 3)), 0));
                } else {
                    // partial chunk (the segment's last): offsets formed here, not held in
                    // registers across the loop
                    uint32_t base = oy;
                    int g4 = 4 * grp;
                    asm volatile("" : "+v"(base), "+v"(g4));
#pragma unroll
                    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int i = 16 * mt + r;
                            const uint32_t o = i + g4 < lim ? base - static_cast<uint32_t>(i * ytokB) : kOOB;
                            yv[4 * mt + r] =
                                __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rYl, o, 0, 0));
                        }
                }
            }
        }

        // decay-weighted Gram tiles M[t][j] = 2^{cs_t - cs_j} dt_j (C_t . B_j), j <= t,
        // held as the transposed product (lane (grp, col): j = 16jt + 4grp + r, t = 16mt + col)
        // (wave w: tiles w, w + 4, w + 8; all operands of a tile are read before its MFMAs;
        // no outputs wanted, e.g. a commit without y: nothing to do)
        const int ntiles = a.y ? kTiles : 0;
        for (int k = wave; k < ntiles; k += 4) {
            const int mt = k < 1 ? 0 : (k < 3 ? 1 : (k < 6 ? 2 : 3));
            const int jt = k - mt * (mt + 1) / 2;
            f32x4 gacc = {0.f, 0.f, 0.f, 0.f};
            if constexpr (F32) {
                f32x4 bq[QN], cq[QN];
#pragma unroll
                for (int q = 0; q < QN; ++q) {
                    bq[q] = f32q(sB, img_idx<QN, true>(jt, q, grp, col));
                    cq[q] = f32q(sC, img_idx<QN, true>(mt, q, grp, col));
                }
#pragma unroll
                for (int q = 0; q < QN; ++q) gacc = mma_f32q(bq[q], cq[q], gacc);
            } else {
                s16x4 bq[QN], cq[QN];
#pragma unroll
                for (int q = 0; q < QN; ++q) {
                    bq[q] = as_s16x4(sB[row_slot<QN>(16 * jt + col, 4 * q + grp)]);
                    cq[q] = as_s16x4(sC[row_slot<QN>(16 * mt + col, 4 * q + grp)]);
                }
                gacc = mma_quads<QN>(bq, cq, gacc);
            }
            const int t = 16 * mt + col;
            const float cst = sCs[t];
            const f32x4 csj = *reinterpret_cast<const f32x4 *>(&sCs[16 * jt + 4 * grp]);
            const f32x4 dtj = *reinterpret_cast<const f32x4 *>(&sDt[16 * jt + 4 * grp]);
            f32x4 m;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int j = 16 * jt + 4 * grp + r;
                const float w = ex2(cst - csj[r]) * dtj[r];
                m[r] = j <= t ? gacc[r] * w : 0.f;
            }
            if constexpr (F32) {
                sM[k * 64 + lane] = __builtin_bit_cast(uint4, m);
            } else {
                s16x4 mh, ml;
                split4(m, mh, ml);
                const uint2 h2 = as_u2(mh), l2 = as_u2(ml);
                sM[k * 64 + lane] = uint4{h2.x, h2.y, l2.x, l2.y};
            }
        }

        // prefix term 2^{cs_t} (C_t . S) for this wave's columns; the state is split
        // into bf16 hi + lo one pair of dstate tiles at a time
        f32x4 Y[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) Y[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (a.y) {
        if constexpr (F32) {
#pragma unroll
            for (int q = 0; q < QN; ++q) {
                f32x4 cq[4];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) cq[mt] = f32q(sC, img_idx<QN, true>(mt, q, grp, col));
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) Y[mt] = mma_f32q(cq[mt], S[q], Y[mt]);
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
#pragma unroll
        for (int q = 0; q < QN; q += 2) {
            if (q + 1 < QN) {
                s16x4 c0[4], c1[4];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    c0[mt] = as_s16x4(sC[row_slot<QN>(16 * mt + col, 4 * q + grp)]);
                    c1[mt] = as_s16x4(sC[row_slot<QN>(16 * mt + col, 4 * q + 4 + grp)]);
                }
                s16x4 h0, l0, h1, l1;
                split4(S[q], h0, l0);
                split4(S[q + 1], h1, l1);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    Y[mt] = mma_k32(c0[mt], c1[mt], h0, h1, Y[mt]);
                    Y[mt] = mma_k32(c0[mt], c1[mt], l0, l1, Y[mt]);
                }
            } else {
                s16x4 h0, l0;
                split4(S[q], h0, l0);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const s16x4 c0 = as_s16x4(sC[row_slot<QN>(16 * mt + col, 4 * q + grp)]);
                    Y[mt] = mma_k16(c0, h0, Y[mt]);
                    Y[mt] = mma_k16(c0, l0, Y[mt]);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
            Y[mt] *= *reinterpret_cast<const f32x4 *>(&sEc[16 * mt + 4 * grp]);
        }
        __syncthreads();   // Gram tiles published
        if (REV && c + 1 < nch) st.issue(c + 1, tid, wave, lane);

        // x operands of this wave's columns (tokens 16jt + 4grp .. +3)
        s16x4 xh[4];
        f32x4 xvf[F32 ? 4 : 1];   // fp32 storage keeps the values; bf16 re-expands xh
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            f32x4 v;
            x_operand<F32>(sXt, jt, wave, lane, xh[jt], v);
            if constexpr (F32) xvf[jt] = v;
        }
        auto xv = [&](int jt) -> f32x4 {
            if constexpr (F32) return xvf[jt];
            else return f32x4{bf16_to_f32(xh[jt][0]), bf16_to_f32(xh[jt][1]),
                              bf16_to_f32(xh[jt][2]), bf16_to_f32(xh[jt][3])};
        };

        if (a.y) {
        // intra-chunk term: y += M x over j <= t
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            if constexpr (F32) {
#pragma unroll
                for (int jt = 0; jt <= mt; ++jt)
                    Y[mt] = mma_f32q(__builtin_bit_cast(f32x4, sM[(mt * (mt + 1) / 2 + jt) * 64 + lane]),
                                     xvf[jt], Y[mt]);
            } else {
#pragma unroll
            for (int jt = 0; jt <= mt; jt += 2) {
                const uint4 v0 = sM[(mt * (mt + 1) / 2 + jt) * 64 + lane];
                const s16x4 h0 = as_s16x4(uint2{v0.x, v0.y}), l0 = as_s16x4(uint2{v0.z, v0.w});
                if (jt + 1 <= mt) {
                    const uint4 v1 = sM[(mt * (mt + 1) / 2 + jt + 1) * 64 + lane];
                    const s16x4 h1 = as_s16x4(uint2{v1.x, v1.y}), l1 = as_s16x4(uint2{v1.z, v1.w});
                    Y[mt] = mma_k32(h0, h1, xh[jt], xh[jt + 1], Y[mt]);
                    Y[mt] = mma_k32(l0, l1, xh[jt], xh[jt + 1], Y[mt]);
                } else if (jt == 0) {
                    Y[mt] = mma_k16(h0, xh[jt], Y[mt]);
                    Y[mt] = mma_k16(l0, xh[jt], Y[mt]);
                } else {
                    // the accumulator comes from 32-deep MFMAs: stay on that shape (zero
                    // upper half) rather than hand it to a 16-deep MFMA
                    constexpr s16x4 z = {0, 0, 0, 0};
                    Y[mt] = mma_k32(h0, z, xh[jt], z, Y[mt]);
                    Y[mt] = mma_k32(l0, z, xh[jt], z, Y[mt]);
                }
            }
            }
        }

        // skip term and store (lane (grp, col): token 16mt + 4grp + r, column p)
        {
            const int lim = st.valid(c);
            const __amdgpu_buffer_rsrc_t rY = rsrc(ybase + st.window(c) * (ytokB / 4));
            float v[16];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const f32x4 out = Y[mt] + skip * xv(mt);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    v[4 * mt + r] = out[r];
                    if constexpr (REV) v[4 * mt + r] += yv[4 * mt + r];
                }
            }
            // full chunks store at the lane's fixed offset plus a scalar offset with no per-row
            // test (the buffer range check does not cover the scalar offset, so a partial
            // chunk takes the tested path).  The four waves write a token row's 256 bytes in
            // 64-byte pieces at different times: the forward pass stores through the cache so
            // the pieces meet in L2 before the line is written back (the reverse pass read the
            // line first, so its nontemporal stores find it there)
            constexpr int ypol = REV ? kNT : 0;
            if (lim == kC) {
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[i]), rY, oyf,
                                                          ysoff(16 * (i >> 2) + (i & 3)), ypol);
            } else {
                // partial chunk: offsets formed here, not held in registers across the loop
                uint32_t base = oy;
                int g4 = 4 * grp;
                asm volatile("" : "+v"(base), "+v"(g4));
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int i = 16 * mt + r;   // + 4grp: this lane's local token
                        const uint32_t o = i + g4 < lim
                                               ? base + static_cast<uint32_t>((REV ? -i : i) * ytokB)
                                               : kOOB;
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[4 * mt + r]), rY, o, 0, ypol);
                    }
            }
        }
        }

        if constexpr (SUB > 0) {
            // several blocks per chunk: carry the state one block at a time and write the
            // state entering each block of this segment (the next segment writes the one
            // entering its own first block)
            constexpr int NSUB = kC / SUB, JPB = SUB / 16;   // blocks, token tiles per block
            const int64_t seg_tokens = st.s1 - st.s0;
            const int64_t nb_seg = (seg_tokens + SUB - 1) / SUB;
            float cs_prev = 0.f;
#pragma unroll
            for (int sb = 0; sb < NSUB; ++sb) {
                if (static_cast<int64_t>(c) * kC + sb * SUB < seg_tokens) {
                    const float cs_end = sCs[(sb + 1) * SUB - 1];
                    const float keepb = ex2(cs_end - cs_prev);
                    cs_prev = cs_end;
                    // this block's tokens, weighted to its end: 2^(cs_end - cs_j) dt_j x_j
                    WOps<F32, T3> wb;
#pragma unroll
                    for (int jt = sb * JPB; jt < (sb + 1) * JPB; ++jt) {
                        const f32x4 csq = *reinterpret_cast<const f32x4 *>(&sCs[16 * jt + 4 * grp]);
                        const f32x4 dtq = *reinterpret_cast<const f32x4 *>(&sDt[16 * jt + 4 * grp]);
                        f32x4 wv;
#pragma unroll
                        for (int r = 0; r < 4; ++r) wv[r] = ex2(cs_end - csq[r]) * dtq[r];
                        w_set(wb, jt, wv * xv(jt));
                    }
                    BtOps<F32> cur;
#pragma unroll
                    for (int q = 0; q < QN; ++q) {
                        bt_read<NS, F32>(cur, F32 ? sBt : sB, q, lane);
                        f32x4 acc = S[q] * keepb;
                        if constexpr (F32) {
#pragma unroll
                            for (int jt = sb * JPB; jt < (sb + 1) * JPB; ++jt)
                                acc = mma_f32q(cur.f[jt], wb.f[jt], acc);
                        } else if constexpr (JPB == 2) {
                            acc = mma_k32(cur.h[2 * sb], cur.h[2 * sb + 1], wb.h[2 * sb], wb.h[2 * sb + 1], acc);
                            acc = mma_k32(cur.h[2 * sb], cur.h[2 * sb + 1], wb.m[2 * sb], wb.m[2 * sb + 1], acc);
                            acc = mma_k32(cur.h[2 * sb], cur.h[2 * sb + 1], wb.l[2 * sb], wb.l[2 * sb + 1], acc);
                        } else {
                            acc = mma_k16(cur.h[sb], wb.h[sb], acc);
                            acc = mma_k16(cur.h[sb], wb.m[sb], acc);
                            acc = mma_k16(cur.h[sb], wb.l[sb], acc);
                        }
                        S[q] = acc;
                        __builtin_amdgcn_sched_barrier(0);
                    }
                    const int64_t blk = static_cast<int64_t>(c) * NSUB + sb + 1;   // S enters it
                    if (blk < nb_seg) {
                        float *dst = emit_base + (emit_first + blk) * a.nheads * (kP * NS);
#pragma unroll
                        for (int q = 0; q < QN; ++q)
                            *reinterpret_cast<f32x4 *>(dst + quad_off(q, grp, p)) = S[q];
                    }
                }
            }
            __syncthreads();   // LDS is rewritten by the next chunk
            continue;
        }

        // carry the state across the chunk (not after the last one unless it is kept)
        if (c + 1 == nch && !a.pool_out) break;
        const float keep = ex2(sCs[kC - 1]);
        WOps<F32, T3> wx;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            w_set(wx, jt, *reinterpret_cast<const f32x4 *>(&sWs[16 * jt + 4 * grp]) * xv(jt));
        BtOps<F32> cur, nxt;
        bt_read<NS, F32>(cur, F32 ? sBt : sB, 0, lane);
#pragma unroll
        for (int q = 0; q < QN; ++q) {
            // the next tile's operands are read while this tile's MFMAs run
            if (q + 1 < QN) bt_read<NS, F32>(nxt, F32 ? sBt : sB, q + 1, lane);
            S[q] = bt_mma(cur, wx, S[q] * keep);
            if (q + 1 < QN) cur = nxt;
            __builtin_amdgcn_sched_barrier(0);
        }
        if (emit_base && c + 1 < nch) {   // the next segment writes the state entering it
            float *dst = emit_base + (emit_first + c + 1) * a.nheads * (kP * NS);
#pragma unroll
            for (int q = 0; q < QN; ++q) *reinterpret_cast<f32x4 *>(dst + quad_off(q, grp, p)) = S[q];
        }
        __syncthreads();   // LDS is rewritten by the next chunk
    }
    if (a.pool_out) {
        float *dst = a.pool_out + (cslot * a.nheads + un.h) * (kP * NS);
#pragma unroll
        for (int q = 0; q < QN; ++q) *reinterpret_cast<f32x4 *>(dst + quad_off(q, grp, p)) = S[q];
    }
}

// ------------------------------------------------------------------ seg_combine
struct CombineArgs {
    float *ws;
    const float *tot;
    float *pool;                 // states entering segment 0 (slot per row), or nullptr: zero
    int64_t units, state_floats; // (row, head) pairs; 64 * N
    int32_t nseg, dirs, nheads;
    int32_t write_final;         // prefill: the final states go back to pool
    int32_t blk_major;           // ws slots as in SeqArgs::blk_major
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

// One thread per 16-byte quad of a (row, head)'s state: the exclusive scans over
// the segments in both directions, in place.
__global__ void __launch_bounds__(256) bdlm_seg_combine_kernel(const CombineArgs c) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int64_t qps = c.state_floats / 4;
    if (i >= c.units * qps) return;
    const int64_t unit = i / qps, e = (i % qps) * 4;
    const int64_t b = unit / c.nheads, h = unit % c.nheads;
    const float *tot = c.tot + unit * c.nseg;
    auto seg = [&](int k) {
        const int64_t slot = c.blk_major ? (b * c.nseg + k) * c.nheads + h : unit * c.nseg + k;
        return reinterpret_cast<f32x4 *>(c.ws + slot * c.dirs * c.state_floats + e);
    };

    float *pst = nullptr;
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    if (c.pool) {
        const int64_t slot = c.use_slots ? c.slots[b] : b;
        pst = c.pool + (slot * c.nheads + h) * c.state_floats + e;
        s = *reinterpret_cast<const f32x4 *>(pst);
    }
    // the recurrence is sequential but its inputs are not: segments go in groups of
    // kG whose loads are all issued before the group's (cheap) arithmetic
    constexpr int kG = 8;
    for (int k0 = 0; k0 < c.nseg; k0 += kG) {
        f32x4 fk[kG];
        float tk[kG];
#pragma unroll
        for (int i = 0; i < kG; ++i)
            if (k0 + i < c.nseg) {
                fk[i] = *seg(k0 + i);
                tk[i] = tot[k0 + i];
            }
#pragma unroll
        for (int i = 0; i < kG; ++i)
            if (k0 + i < c.nseg) {
                *seg(k0 + i) = s;
                s = s * ex2(tk[i]) + fk[i];
            }
    }
    if (c.write_final) *reinterpret_cast<f32x4 *>(pst) = s;
    if (c.dirs == 2) {
        f32x4 r = {0.f, 0.f, 0.f, 0.f};
        for (int k0 = c.nseg - 1; k0 >= 0; k0 -= kG) {
            f32x4 rk[kG];
            float tk[kG];
#pragma unroll
            for (int i = 0; i < kG; ++i)
                if (k0 - i >= 0) {
                    rk[i] = *(seg(k0 - i) + c.state_floats / 4);
                    tk[i] = tot[k0 - i];
                }
#pragma unroll
            for (int i = 0; i < kG; ++i)
                if (k0 - i >= 0) {
                    *(seg(k0 - i) + c.state_floats / 4) = r;
                    r = r * ex2(tk[i]) + rk[i];
                }
        }
    }
}

// ------------------------------------------------------------------ host side
template <int NS, bool F32>
hipError_t state_launch(const SeqArgs &k, bool both, unsigned grid, hipStream_t s) {
    if (both)
        hipLaunchKernelGGL((bdlm_seg_state_kernel<NS, F32, true>), dim3(grid), dim3(kThreads), 0, s, k);
    else
        hipLaunchKernelGGL((bdlm_seg_state_kernel<NS, F32, false>), dim3(grid), dim3(kThreads), 0, s, k);
    return hipGetLastError();
}
template <int NS, bool F32>
hipError_t out_launch(const SeqArgs &k, bool rev, unsigned grid, hipStream_t s) {
    if (rev)
        hipLaunchKernelGGL((bdlm_seg_out_kernel<NS, F32, true, 0>), dim3(grid), dim3(kThreads), 0, s,
                           k);
    else if (k.pool_out || k.emit)   // the carried state is written out
        hipLaunchKernelGGL((bdlm_seg_out_kernel<NS, F32, false, 0, true>), dim3(grid), dim3(kThreads),
                           0, s, k);
    else
        hipLaunchKernelGGL((bdlm_seg_out_kernel<NS, F32, false, 0>), dim3(grid), dim3(kThreads), 0,
                           s, k);
    return hipGetLastError();
}
template <int NS, bool F32>
hipError_t out_sub_launch(const SeqArgs &k, int sub, unsigned grid, hipStream_t s) {
    if (sub == 16)
        hipLaunchKernelGGL((bdlm_seg_out_kernel<NS, F32, false, 16>), dim3(grid), dim3(kThreads), 0,
                           s, k);
    else
        hipLaunchKernelGGL((bdlm_seg_out_kernel<NS, F32, false, 32>), dim3(grid), dim3(kThreads), 0,
                           s, k);
    return hipGetLastError();
}

template <bool F32>
hipError_t run_state(int ns, const SeqArgs &k, bool both, unsigned grid, hipStream_t s) {
    switch (ns) {
        case 16: return state_launch<16, F32>(k, both, grid, s);
        case 32: return state_launch<32, F32>(k, both, grid, s);
        case 64: return state_launch<64, F32>(k, both, grid, s);
        case 128: return state_launch<128, F32>(k, both, grid, s);
        default: return hipErrorInvalidValue;
    }
}
template <bool F32>
hipError_t run_out_sub(int ns, const SeqArgs &k, int sub, unsigned grid, hipStream_t s) {
    switch (ns) {
        case 16: return out_sub_launch<16, F32>(k, sub, grid, s);
        case 32: return out_sub_launch<32, F32>(k, sub, grid, s);
        case 64: return out_sub_launch<64, F32>(k, sub, grid, s);
        case 128: return out_sub_launch<128, F32>(k, sub, grid, s);
        default: return hipErrorInvalidValue;
    }
}
template <bool F32>
hipError_t run_out(int ns, const SeqArgs &k, bool rev, unsigned grid, hipStream_t s) {
    switch (ns) {
        case 16: return out_launch<16, F32>(k, rev, grid, s);
        case 32: return out_launch<32, F32>(k, rev, grid, s);
        case 64: return out_launch<64, F32>(k, rev, grid, s);
        case 128: return out_launch<128, F32>(k, rev, grid, s);
        default: return hipErrorInvalidValue;
    }
}

SeqArgs seq_args(const LaunchArgs &a, int64_t T, const SeqPlan &pl, void *ws) {
    SeqArgs k;
    k.x = a.x;
    k.dt = a.dt;
    k.Bm = a.Bm;
    k.Cm = a.Cm;
    k.A = a.A;
    k.skip = a.D;
    k.y = a.y;
    k.ws = static_cast<float *>(ws);
    k.tot = ws ? static_cast<float *>(ws) + pl.state_bytes / 4 : nullptr;
    k.xs_b = a.xs_b;
    k.xs_t = a.xs_t;
    k.xs_h = a.xs_h;
    k.dts_b = a.dts_b;
    k.dts_t = a.dts_t;
    k.bcs_b = a.bcs_b;
    k.bcs_t = a.bcs_t;
    k.bcs_g = a.bcs_g;
    k.T = T;
    k.S = pl.seg_len;
    k.nseg = static_cast<int32_t>(pl.nseg);
    k.dirs = pl.dirs;
    k.nheads = a.nheads;
    k.heads_per_group = a.nheads / a.ngroups;
    k.zero_init = 1;
    k.blk_major = 0;
    k.pool_in = nullptr;
    k.pool_out = nullptr;
    k.cstride = kC;
    k.emit = nullptr;
    k.emit_blocks = 0;
    k.use_slots = a.slots ? 1 : 0;
    for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i)
        k.slots[i] = (a.slots && i < a.batch) ? a.slots[i] : 0;
    const int64_t grid = static_cast<int64_t>(a.batch) * a.nheads * pl.nseg;
    k.xcd_remap = grid % 8 == 0 ? 1 : 0;
    return k;
}

hipError_t combine(const LaunchArgs &a, const SeqPlan &pl, const SeqArgs &k, float *pool,
                   bool write_final, hipStream_t s) {
    CombineArgs c;
    c.ws = k.ws;
    c.tot = k.tot;
    c.pool = pool;
    c.write_final = write_final && pool ? 1 : 0;
    c.blk_major = k.blk_major;
    c.units = static_cast<int64_t>(a.batch) * a.nheads;
    c.state_floats = static_cast<int64_t>(kP) * a.dstate;
    c.nseg = static_cast<int32_t>(pl.nseg);
    c.dirs = pl.dirs;
    c.nheads = a.nheads;
    c.use_slots = a.slots ? 1 : 0;
    for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i)
        c.slots[i] = (a.slots && i < a.batch) ? a.slots[i] : 0;
    const int64_t threads = c.units * (c.state_floats / 4);
    const unsigned grid = static_cast<unsigned>((threads + 255) / 256);
    hipLaunchKernelGGL(bdlm_seg_combine_kernel, dim3(grid), dim3(256), 0, s, c);
    return hipGetLastError();
}

}  // namespace

int launch_full_window(const LaunchArgs &a, int64_t T, void *ws, void *stream) {
    if (a.batch == 0 || T == 0) return BDLM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const SeqPlan pl = seq_plan(a.batch, a.nheads, a.dstate, T, 2);
    SeqArgs k = seq_args(a, T, pl, pl.nseg > 1 ? ws : nullptr);
    const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(a.batch) * a.nheads * pl.nseg);
    const bool f32 = !a.bf16;
    if (pl.nseg > 1) {
        // local states, then the states entering every segment
        if ((f32 ? run_state<true>(a.dstate, k, true, grid, s)
                 : run_state<false>(a.dstate, k, true, grid, s)) != hipSuccess)
            return BDLM_E_LAUNCH;
        if (combine(a, pl, k, nullptr, false, s) != hipSuccess) return BDLM_E_LAUNCH;
        k.zero_init = 0;
    }
    k.skip = a.D;
    if ((f32 ? run_out<true>(a.dstate, k, false, grid, s) : run_out<false>(a.dstate, k, false, grid, s)) !=
        hipSuccess)
        return BDLM_E_LAUNCH;
    k.skip = a.D_rev;
    if ((f32 ? run_out<true>(a.dstate, k, true, grid, s) : run_out<false>(a.dstate, k, true, grid, s)) !=
        hipSuccess)
        return BDLM_E_LAUNCH;
    return BDLM_OK;
}

int launch_prefill(const LaunchArgs &a, int64_t T, void *ws, void *stream, const SeqPlan *plan) {
    if (a.batch == 0 || T == 0) return BDLM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const SeqPlan pl = plan ? *plan : seq_plan(a.batch, a.nheads, a.dstate, T, 1);
    SeqArgs k = seq_args(a, T, pl, ws);
    const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(a.batch) * a.nheads * pl.nseg);
    const bool f32 = !a.bf16;
    if ((f32 ? run_state<true>(a.dstate, k, false, grid, s)
             : run_state<false>(a.dstate, k, false, grid, s)) != hipSuccess)
        return BDLM_E_LAUNCH;
    // the cached states enter segment 0; the final states go back to the cache
    if (combine(a, pl, k, a.h_pool, true, s) != hipSuccess) return BDLM_E_LAUNCH;
    if (a.y) {
        k.zero_init = 0;
        k.skip = a.D;
        if ((f32 ? run_out<true>(a.dstate, k, false, grid, s)
                 : run_out<false>(a.dstate, k, false, grid, s)) != hipSuccess)
            return BDLM_E_LAUNCH;
    }
    return BDLM_OK;
}

int launch_boundary_states(const LaunchArgs &a, int64_t nblocks, const float *s_init,
                           float *s_out, void *ws, void *stream) {
    if (a.batch == 0 || nblocks == 0) return BDLM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // segments of G whole blocks: local segment states (seg_state), the states entering
    // the segments (seg_combine), then one sweep per segment, a block per chunk, that
    // writes every block's entering state (and the forward outputs if wanted)
    const BoundaryPlan bp = boundary_plan(a.batch, a.nheads, a.dstate, nblocks, a.L);
    SeqPlan pl;
    pl.seg_len = bp.blocks_per_seg * a.L;
    pl.nseg = bp.nseg;
    pl.dirs = 1;
    pl.state_bytes = bp.state_bytes;
    pl.total_bytes = bp.total_bytes;
    SeqArgs k = seq_args(a, nblocks * a.L, pl, bp.nseg > 1 ? ws : nullptr);
    const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(a.batch) * a.nheads * bp.nseg);
    const bool f32 = !a.bf16;
    if (bp.nseg > 1 || s_init) {
        if (bp.nseg > 1 && (f32 ? run_state<true>(a.dstate, k, false, grid, s)
                                : run_state<false>(a.dstate, k, false, grid, s)) != hipSuccess)
            return BDLM_E_LAUNCH;
        if (bp.nseg == 1) {   // one segment: its entering state is s_init itself
            k.pool_in = s_init;
            k.use_slots = 0;
        } else {
            if (combine(a, pl, k, const_cast<float *>(s_init), false, s) != hipSuccess)
                return BDLM_E_LAUNCH;
            k.zero_init = 0;
        }
    }
    k.emit = s_out;
    k.emit_blocks = nblocks;
    k.skip = a.D;
    hipError_t e;
    if (a.L == 16 || a.L == 32) {   // 64-token chunks carrying the state block by block
        k.cstride = kC;
        e = f32 ? run_out_sub<true>(a.dstate, k, a.L, grid, s)
                : run_out_sub<false>(a.dstate, k, a.L, grid, s);
    } else {                        // one block per chunk
        k.cstride = a.L;
        e = f32 ? run_out<true>(a.dstate, k, false, grid, s) : run_out<false>(a.dstate, k, false, grid, s);
    }
    if (e != hipSuccess) return BDLM_E_LAUNCH;
    return BDLM_OK;
}

// One segment per row: a block of any length from the cached state.
static SeqArgs block_args(const LaunchArgs &a) {
    SeqPlan pl;
    pl.seg_len = a.L;
    pl.nseg = 1;
    pl.dirs = 1;
    pl.state_bytes = 0;
    pl.total_bytes = 0;
    return seq_args(a, a.L, pl, nullptr);
}

int launch_block_long(const LaunchArgs &fwd, const LaunchArgs &rev, bool commit, bool want_y,
                      void *stream) {
    if (fwd.batch == 0 || fwd.L == 0) return BDLM_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(fwd.batch) * fwd.nheads);
    const bool f32 = !fwd.bf16;
    // forward from the cached state (a commit writes the final state back in place)
    SeqArgs k = block_args(fwd);
    k.pool_in = fwd.h_pool;
    k.pool_out = commit ? fwd.h_pool : nullptr;
    k.y = want_y ? fwd.y : nullptr;
    k.skip = fwd.D;
    if (k.y || k.pool_out) {
        if ((f32 ? run_out<true>(fwd.dstate, k, false, grid, s)
                 : run_out<false>(fwd.dstate, k, false, grid, s)) != hipSuccess)
            return BDLM_E_LAUNCH;
    }
    if (!want_y) return BDLM_OK;
    // reverse inside the block from zero, added onto y
    SeqArgs r = block_args(rev);
    r.y = fwd.y;
    r.skip = rev.D_rev;
    if ((f32 ? run_out<true>(rev.dstate, r, true, grid, s)
             : run_out<false>(rev.dstate, r, true, grid, s)) != hipSuccess)
        return BDLM_E_LAUNCH;
    return BDLM_OK;
}

}  // namespace bdlm
