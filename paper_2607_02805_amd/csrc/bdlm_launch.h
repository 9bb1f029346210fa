// Internal interface between the host entry points (bdlm_api.cpp) and the HIP
// kernels (bdlm_scan.hip).  Plain C++; no HIP types.
#pragma once

#include <stdint.h>

#include "bdlm.h"

namespace bdlm {

struct LaunchArgs {
    const void *x, *dt, *Bm, *Cm;
    const float *A, *D, *D_rev;
    float *h_pool;   // read only for a step, updated in place by a commit
    float *y;        // step: required; commit: optional (NULL skips y_clean)
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int32_t batch, nheads, ngroups, L, dstate;
    int32_t bf16;          // activation storage: 1 bf16, 0 fp32
    const int32_t *slots;  // host [batch] or NULL (identity)
};

// Enqueue one block step (commit == false) or one commit (commit == true).
// Arguments are already validated.  Returns BDLM_OK or BDLM_E_LAUNCH.
int launch_block(const LaunchArgs &a, bool commit, void *stream);

// Commit of the clean block (clean; clean.y: its outputs, or nullptr) followed by the first
// denoising step of the next block (next's inputs, outputs into y_next) from the updated
// state, for blocks of at most 64 tokens (next has clean's shapes, slots and parameters).
// A bf16 block of at most 32 tokens is one launch that reads the state once; otherwise a
// commit launch and a step launch.
int launch_commit_step(const LaunchArgs &clean, const LaunchArgs &next, float *y_next,
                       void *stream);

// A step (or commit) of a block of at most 64 tokens whose reverse branch has inputs of
// its own: the forward branch of `fwd` from the cached state (skip fwd.D) plus the
// reverse branch of `rev` (skip rev.D_rev) into y; a commit updates the state from
// `fwd`.  A bf16 step of at most 32 tokens is one launch computing both branches;
// otherwise the forward launch stores y and a reverse launch adds onto it.  want_y
// false (commit only): no outputs, no reverse launch.
int launch_block_pair(const LaunchArgs &fwd, const LaunchArgs &rev, bool commit, bool want_y,
                      void *stream);

// A step (or commit) of a block of at most 32 tokens with the convolution part of the
// boundary state, bf16 inputs before the convolution: the convolution runs while each
// launch stages its inputs (forward launch from the cached rows conv_pool, then the
// reverse launch zero-padded past the block), with no workspace.  The forward launch
// stores y (none when want_y is false) and a commit updates the state; the reverse
// launch adds onto y.  conv_pool is only read: a commit's new cache rows are written
// by the caller afterwards.
int launch_conv_fused(const LaunchArgs &a, const float *w, const float *bias, const float *conv_pool,
                      bool commit, bool want_y, void *stream);

// How the sequence kernels cut T tokens into segments (one workgroup per batch row,
// head and segment) and the device workspace they need: per (row, head, segment)
// `dirs` states of 64 x dstate fp32, then one fp32 log-decay, rounded up to 256
// bytes.  Segments are sized for about 2048 workgroups, at least 256 tokens each.
struct SeqPlan {
    int64_t seg_len, nseg;
    int32_t dirs;
    int64_t state_bytes, total_bytes;
};
inline SeqPlan seq_plan(int64_t batch, int64_t nheads, int64_t dstate, int64_t T, int32_t dirs) {
    SeqPlan p;
    p.dirs = dirs;
    const int64_t units = batch * nheads;
    const int64_t want = units >= 2048 ? 1 : (2048 + units - 1) / units;
    int64_t S = (T + want - 1) / want;
    S = (S + 63) / 64 * 64;
    if (S < 256) S = 256;
    p.seg_len = S;
    p.nseg = T > 0 ? (T + S - 1) / S : 1;
    p.state_bytes = units * p.nseg * dirs * int64_t(BDLM_HEADDIM) * dstate * 4;
    p.total_bytes = p.state_bytes + (units * p.nseg * 4 + 255) / 256 * 256;
    return p;
}
// Workspace bytes of a full window (none when the window is one segment) and of a
// prefill.
inline int64_t full_window_workspace(int64_t batch, int64_t nheads, int64_t dstate, int64_t T) {
    if (batch == 0 || T == 0) return 0;
    const SeqPlan p = seq_plan(batch, nheads, dstate, T, 2);
    return p.nseg > 1 ? p.total_bytes : 0;
}
inline int64_t prefill_workspace(int64_t batch, int64_t nheads, int64_t dstate, int64_t T) {
    if (batch == 0 || T == 0) return 0;
    const int64_t full = seq_plan(batch, nheads, dstate, T, 1).total_bytes;
    if (batch <= BDLM_MAX_SLOT_ROWS) return full;
    // a slot-mapped call runs in launches of BDLM_MAX_SLOT_ROWS rows, each planned (and
    // reusing the workspace from its start) on its own
    const int64_t chunk = seq_plan(BDLM_MAX_SLOT_ROWS, nheads, dstate, T, 1).total_bytes;
    const int64_t tail_rows = batch % BDLM_MAX_SLOT_ROWS;
    const int64_t tail = tail_rows ? seq_plan(tail_rows, nheads, dstate, T, 1).total_bytes : 0;
    return full > chunk ? (full > tail ? full : tail) : (chunk > tail ? chunk : tail);
}

// Full-window bidirectional scan over T tokens (a.L is ignored): forward pass,
// then reverse pass adding into a.y.  ws: full_window_workspace bytes.
int launch_full_window(const LaunchArgs &a, int64_t T, void *ws, void *stream);

// Forward scan over T tokens continuing the states in a.h_pool (via a.slots),
// writing them back; a.y (optional) receives the forward outputs.
// ws: prefill_workspace bytes, or plan->total_bytes when a plan is given (nullptr: the
// standard plan seq_plan(a.batch, a.nheads, a.dstate, T, 1)).
int launch_prefill(const LaunchArgs &a, int64_t T, void *ws, void *stream,
                   const SeqPlan *plan = nullptr);

// A prefill plan whose workspace fits in cap bytes: the standard plan if it fits, else
// fewer and longer segments (the same computation with fewer workgroups).  False if
// even one segment per row and head needs more than cap.
inline bool prefill_plan_capped(int64_t batch, int64_t nheads, int64_t dstate, int64_t T,
                                int64_t cap, SeqPlan *out) {
    SeqPlan p = seq_plan(batch, nheads, dstate, T, 1);
    if (p.total_bytes > cap) {
        const int64_t units = batch * nheads;
        const int64_t per_seg = units * int64_t(BDLM_HEADDIM) * dstate * 4;
        int64_t nseg = (cap - (units * p.nseg * 4 + 255) / 256 * 256) / per_seg;
        if (nseg < 1) return false;
        int64_t S = (T + nseg - 1) / nseg;
        S = (S + 63) / 64 * 64;
        if (S < 256) S = 256;
        p.seg_len = S;
        p.nseg = (T + S - 1) / S;
        p.state_bytes = units * p.nseg * int64_t(BDLM_HEADDIM) * dstate * 4;
        p.total_bytes = p.state_bytes + (units * p.nseg * 4 + 255) / 256 * 256;
        if (p.total_bytes > cap) return false;
    }
    *out = p;
    return true;
}

// The library's own device scratch of the no-allocation prefill: BDLM_SCRATCH_BYTES,
// 256-byte aligned, one array per device (its address on the current device, looked
// up once per device).  BDLM_OK, or BDLM_E_LAUNCH if the runtime cannot resolve it.
int scratch_pointer(void **out);

// States entering every block of a clean sequence of nblocks blocks of a.L tokens:
// s_out[(row * nblocks + k) * nheads + head] (pool layout) = the forward state after
// blocks 0 .. k-1, starting from s_init[row * nheads + head] (nullptr: zero).  a.y
// (optional) receives the forward outputs of the sequence.  ws: boundary_workspace
// bytes.  The blocks go in segments of blocks_per_seg (sized for ~4096 workgroups);
// the workspace holds one state and one log-decay per (row, head, segment).
struct BoundaryPlan {
    int64_t blocks_per_seg, nseg, state_bytes, total_bytes;
};
inline BoundaryPlan boundary_plan(int64_t batch, int64_t nheads, int64_t dstate, int64_t nblocks,
                                  int64_t L) {
    BoundaryPlan p;
    const int64_t units = batch * nheads;
    const int64_t want = units >= 4096 ? 1 : (4096 + units - 1) / units;   // segments per row
    p.blocks_per_seg = (nblocks + want - 1) / want;
    if (p.blocks_per_seg * L < 256) p.blocks_per_seg = (256 + L - 1) / L;   // >= 256 tokens
    if (L == 16 || L == 32) {   // whole 64-token chunks per segment
        const int64_t per = 64 / L;
        p.blocks_per_seg = (p.blocks_per_seg + per - 1) / per * per;
    }
    if (p.blocks_per_seg > nblocks) p.blocks_per_seg = nblocks > 0 ? nblocks : 1;
    p.nseg = nblocks > 0 ? (nblocks + p.blocks_per_seg - 1) / p.blocks_per_seg : 1;
    p.state_bytes = units * p.nseg * int64_t(BDLM_HEADDIM) * dstate * 4;
    p.total_bytes = p.state_bytes + (units * p.nseg * 4 + 255) / 256 * 256;
    return p;
}
int launch_boundary_states(const LaunchArgs &a, int64_t nblocks, const float *s_init,
                           float *s_out, void *ws, void *stream);
inline int64_t boundary_workspace(int64_t batch, int64_t nheads, int64_t dstate, int64_t nblocks,
                                  int64_t L) {
    if (batch == 0 || nblocks == 0 || L == 0) return 0;
    const BoundaryPlan p = boundary_plan(batch, nheads, dstate, nblocks, L);
    return p.nseg > 1 ? p.total_bytes : 0;   // one segment: a single sweep, no workspace
}

// A block of any length (a.L) as one segment per row: the forward branch from the
// cached state (fwd's inputs, skip fwd.D) and, if want_y, the reverse branch from zero
// (rev's inputs, skip rev.D_rev) added into fwd.y.  commit: the final forward state is
// written back to fwd.h_pool in place.  fwd and rev share shapes and slots.
int launch_block_long(const LaunchArgs &fwd, const LaunchArgs &rev, bool commit, bool want_y,
                      void *stream);

// Blocks of 65 to 256 tokens with bf16 activations and one input set for both branches:
// one launch in masked-matrix form, one workgroup per (row, head) (bdlm_mask.hip).
bool long_masked_fits(const LaunchArgs &a);
int launch_long_masked(const LaunchArgs &a, bool commit, bool want_y, void *stream);
// A long block's step or commit with one input set: launch_long_masked where it fits,
// else launch_block_long.
int launch_block_long_shared(const LaunchArgs &a, bool commit, bool want_y, void *stream);

// The convolution part of the boundary state, then the block step (commit: the
// commit) on the convolved inputs: a.x / a.Bm / a.Cm are the pre-convolution inputs,
// conv_pool [nslots][3][channels] the cached input rows (a commit replaces them).
// ws: conv_workspace bytes (fp32 convolved x, B, C for both branches and dt).
int launch_conv_block(const LaunchArgs &a, const float *w, const float *bias, float *conv_pool,
                      bool commit, void *ws, void *stream);
inline int64_t conv_workspace(int64_t batch, int64_t L, int64_t nheads, int64_t ngroups,
                              int64_t dstate) {
    const int64_t HP = nheads * BDLM_HEADDIM, GN = ngroups * dstate;
    return (batch * L * (2 * HP + 4 * GN + nheads) * 4 + 255) / 256 * 256;
}

// Permute nstates states between row-major [64][dstate] and the pool layout.
// Gated RMS normalisation of a mixer output: out = w * g / sqrt(mean_group(g^2) + eps),
// g = y * silu(z), per token over nheads * 64 channels in ngroups groups of whole heads.
// y, out fp32 [batch][len][nheads * 64] contiguous (out may be y); z [batch][len][channels]
// with strides zs_b, zs_t (elements), unit channel stride; nheads <= 256.
struct NormLaunch {
    const float *y;
    const void *z;
    const float *w;
    float *out;
    int64_t zs_b, zs_t, batch, len, nheads, ngroups;
    int32_t bf16;
    float eps;
};
int launch_gated_rmsnorm(const NormLaunch &n, void *stream);

int launch_state_permute(const float *src, float *dst, int64_t nstates, int64_t dstate,
                         bool to_pool, void *stream);

// Zero nreset states of state_elems floats each (slots NULL: all nslots).
int launch_reset(float *h_pool, int64_t nslots, int64_t state_elems, const int32_t *slots,
                 int64_t nreset, void *stream);

}  // namespace bdlm
