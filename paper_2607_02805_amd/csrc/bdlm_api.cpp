// bdlm_api.cpp -- the C ABI of libbdlm (declared in include/bdlm.h): argument
// checks on the host, cache bookkeeping, and dispatch to the HIP launchers.
// Every check runs before anything is enqueued, so every error path can be
// exercised without a GPU.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "bdlm.h"
#include "bdlm_launch.h"

namespace {

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int64_t elem_size(int32_t dt) { return dt == BDLM_DTYPE_BF16 ? 2 : 4; }

// Checks of the descriptor alone.  max_len: the longest block_len the entry point
// accepts.
int check_desc(const bdlm_desc_t *d, int64_t max_len) {
    if (!d) return BDLM_E_NULL;
    if (d->in_dtype != BDLM_DTYPE_F32 && d->in_dtype != BDLM_DTYPE_BF16) return BDLM_E_DTYPE;
    if (d->reserved != 0) return BDLM_E_DTYPE;
    if (d->batch < 0 || d->nheads <= 0 || d->ngroups <= 0 || d->block_len < 0) return BDLM_E_SHAPE;
    if (d->headdim != BDLM_HEADDIM) return BDLM_E_SHAPE;
    if (d->dstate != 16 && d->dstate != 32 && d->dstate != 64 && d->dstate != 128)
        return BDLM_E_SHAPE;
    if (d->block_len > max_len) return BDLM_E_SHAPE;
    if (d->nheads % d->ngroups != 0) return BDLM_E_SHAPE;
    // every launch grid stays within 32 bits
    constexpr int64_t kMaxRows = int64_t(1) << 22;
    if (d->batch > kMaxRows || d->nheads > kMaxRows || d->batch * d->nheads > kMaxRows)
        return BDLM_E_SHAPE;
    for (int i = 0; i < 3; ++i)
        if (d->x_stride[i] < 0 || d->bc_stride[i] < 0) return BDLM_E_SHAPE;
    if (d->dt_stride[0] < 0 || d->dt_stride[1] < 0) return BDLM_E_SHAPE;
    return BDLM_OK;
}

// Checks shared by every entry point that takes activations.
// need_pool: the call reads or writes a state pool (h_pool, nslots and slot_idx
// are checked).
int check_common(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                 const void *B, const void *C, const float *D, const float *D_rev,
                 const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                 int64_t max_len = BDLM_MAX_BLOCK_LEN, bool need_pool = true) {
    const int rc = check_desc(d, max_len);
    if (rc != BDLM_OK) return rc;
    if (need_pool && nslots <= 0) return BDLM_E_SHAPE;
    if (need_pool && nslots > (int64_t(1) << 40) / (d->nheads * BDLM_HEADDIM * d->dstate))
        return BDLM_E_SHAPE;
    // With no token to read, the activation pointers may be NULL (an empty tensor
    // can have no storage).
    const bool empty = d->batch == 0 || d->block_len == 0;
    if (!empty && (!x || !dt || !B || !C)) return BDLM_E_NULL;
    if (!A || !D || !D_rev || (need_pool && !h_pool)) return BDLM_E_NULL;

    // x, B and C are read in 16-byte vectors: base pointers 16-byte aligned and
    // every stride a whole number of 16-byte units.
    const int64_t es = elem_size(d->in_dtype);
    const int64_t vec = 16 / es;
    if (!aligned(x, 16) || !aligned(B, 16) || !aligned(C, 16)) return BDLM_E_ALIGN;
    if (!aligned(dt, es)) return BDLM_E_ALIGN;
    for (int i = 0; i < 3; ++i)
        if (d->bc_stride[i] % vec != 0 || d->x_stride[i] % vec != 0) return BDLM_E_ALIGN;
    if (!aligned(A, 4) || !aligned(D, 4) || !aligned(D_rev, 4)) return BDLM_E_ALIGN;
    if (!need_pool) return BDLM_OK;
    if (!aligned(h_pool, 16)) return BDLM_E_ALIGN;

    if (slot_idx) {
        for (int64_t b = 0; b < d->batch; ++b)
            if (slot_idx[b] < 0 || slot_idx[b] >= nslots) return BDLM_E_SLOT;
    } else if (d->batch > nslots) {
        return BDLM_E_SLOT;
    }
    return BDLM_OK;
}

// The sequence kernels address a 64-token chunk with 32-bit byte offsets from a
// per-chunk base: every per-token stride (and y's, nheads x 64 floats) stays below
// 16 MiB.
int check_seq_strides(const bdlm_desc_t *d) {
    constexpr int64_t kMaxRow = int64_t(1) << 24;
    const int64_t es = elem_size(d->in_dtype);
    if (d->x_stride[1] * es > kMaxRow || d->bc_stride[1] * es > kMaxRow ||
        d->dt_stride[1] * es > kMaxRow || d->nheads * BDLM_HEADDIM * 4 > kMaxRow)
        return BDLM_E_SHAPE;
    return BDLM_OK;
}

bdlm::LaunchArgs make_args(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                           const void *B, const void *C, const float *D, const float *D_rev,
                           float *h_pool, const int32_t *slot_idx, float *y) {
    bdlm::LaunchArgs a;
    a.x = x;
    a.dt = dt;
    a.Bm = B;
    a.Cm = C;
    a.A = A;
    a.D = D;
    a.D_rev = D_rev;
    a.h_pool = h_pool;
    a.y = y;
    a.xs_b = d->x_stride[0];
    a.xs_t = d->x_stride[1];
    a.xs_h = d->x_stride[2];
    a.dts_b = d->dt_stride[0];
    a.dts_t = d->dt_stride[1];
    a.bcs_b = d->bc_stride[0];
    a.bcs_t = d->bc_stride[1];
    a.bcs_g = d->bc_stride[2];
    a.batch = static_cast<int32_t>(d->batch);
    a.nheads = static_cast<int32_t>(d->nheads);
    a.ngroups = static_cast<int32_t>(d->ngroups);
    a.L = static_cast<int32_t>(d->block_len);
    a.dstate = static_cast<int32_t>(d->dstate);
    a.bf16 = d->in_dtype == BDLM_DTYPE_BF16 ? 1 : 0;
    a.slots = slot_idx;
    return a;
}

// Rows [r0, r0 + n) of a call as a call of its own: the activations and outputs
// advanced by r0 rows (y_row floats of output per row), the slot table by r0 entries.
bdlm::LaunchArgs rows_of(const bdlm::LaunchArgs &a, int64_t r0, int64_t n, int64_t y_row) {
    bdlm::LaunchArgs s = a;
    const int64_t es = a.bf16 ? 2 : 4;
    auto adv = [&](const void *p, int64_t elems) {
        return p ? static_cast<const void *>(static_cast<const char *>(p) + elems * es) : p;
    };
    s.x = adv(a.x, r0 * a.xs_b);
    s.dt = adv(a.dt, r0 * a.dts_b);
    s.Bm = adv(a.Bm, r0 * a.bcs_b);
    s.Cm = adv(a.Cm, r0 * a.bcs_b);
    if (a.y) s.y = a.y + r0 * y_row;
    if (a.slots) s.slots = a.slots + r0;
    s.batch = static_cast<int32_t>(n);
    return s;
}

// The kernels take an explicit slot table by value, BDLM_MAX_SLOT_ROWS rows per launch:
// a call with a longer table runs as consecutive launches over row ranges (on one
// stream, in order, so a workspace is reused safely).  launch(args...) receives the
// sliced arguments.
template <class F>
int by_row_chunks(const bdlm::LaunchArgs &a, int64_t y_row, F &&launch) {
    if (!a.slots || a.batch <= BDLM_MAX_SLOT_ROWS) return launch(a);
    for (int64_t r0 = 0; r0 < a.batch; r0 += BDLM_MAX_SLOT_ROWS) {
        const int64_t n = std::min<int64_t>(BDLM_MAX_SLOT_ROWS, a.batch - r0);
        const int rc = launch(rows_of(a, r0, n, y_row));
        if (rc != BDLM_OK) return rc;
    }
    return BDLM_OK;
}

// Output floats per batch row of a block (or sequence) of len tokens.
int64_t y_row_floats(const bdlm_desc_t *d, int64_t len) { return len * d->nheads * BDLM_HEADDIM; }

}  // namespace

extern "C" {

int bdlm_abi_version(void) { return BDLM_ABI_VERSION; }

const char *bdlm_strerror(int status) {
    switch (status) {
        case BDLM_OK: return "ok";
        case BDLM_E_NULL: return "a required pointer is NULL";
        case BDLM_E_SHAPE: return "unsupported or inconsistent sizes";
        case BDLM_E_DTYPE: return "unknown activation dtype or nonzero reserved field";
        case BDLM_E_ALIGN: return "pointer or stride breaks the alignment contract";
        case BDLM_E_OFFSET: return "cache slot does not hold the expected number of blocks";
        case BDLM_E_SLOT: return "slot index out of range or repeated in a commit";
        case BDLM_E_LAUNCH: return "HIP launch failed";
        case BDLM_E_WORKSPACE: return "workspace missing or smaller than required";
        default: return "unknown status";
    }
}

int bdlm_desc_init(bdlm_desc_t *d, int64_t batch, int64_t nheads, int64_t headdim, int64_t dstate,
                   int64_t ngroups, int64_t block_len, int32_t in_dtype) {
    if (!d) return BDLM_E_NULL;
    memset(d, 0, sizeof *d);
    d->batch = batch;
    d->nheads = nheads;
    d->headdim = headdim;
    d->dstate = dstate;
    d->ngroups = ngroups;
    d->block_len = block_len;
    d->in_dtype = in_dtype;
    d->x_stride[2] = headdim;
    d->x_stride[1] = nheads * headdim;
    d->x_stride[0] = block_len * nheads * headdim;
    d->dt_stride[1] = nheads;
    d->dt_stride[0] = block_len * nheads;
    d->bc_stride[2] = dstate;
    d->bc_stride[1] = ngroups * dstate;
    d->bc_stride[0] = block_len * ngroups * dstate;
    return BDLM_OK;
}

// Blocks longer than BDLM_MAX_BLOCK_LEN run on the sequence kernels: their strides
// are limited as for the sequence entry points.
static int check_long_block(const bdlm_desc_t *d) {
    return d->block_len > BDLM_MAX_BLOCK_LEN ? check_seq_strides(d) : BDLM_OK;
}

int bdlm_check_block_step(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                          const void *B, const void *C, const float *D, const float *D_rev,
                          const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                          const float *y) {
    int rc = check_common(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx,
                          BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    rc = check_long_block(d);
    if (rc != BDLM_OK) return rc;
    if (!y && d->batch != 0 && d->block_len != 0) return BDLM_E_NULL;
    if (!aligned(y, 16)) return BDLM_E_ALIGN;
    return BDLM_OK;
}

static int check_books(const bdlm_desc_t *d, const int32_t *slot_idx, const int64_t *n_committed,
                       const int64_t *n_blocks, int64_t expected_block_index) {
    if (!n_committed || !n_blocks) return BDLM_E_NULL;
    if (slot_idx && d->batch > 1) {   // the rows of a commit write distinct slots
        std::vector<int32_t> sorted(slot_idx, slot_idx + d->batch);
        std::sort(sorted.begin(), sorted.end());
        if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end()) return BDLM_E_SLOT;
    }
    for (int64_t b = 0; b < d->batch; ++b) {
        const int64_t s = slot_idx ? slot_idx[b] : b;
        if (expected_block_index >= 0 && n_blocks[s] != expected_block_index) return BDLM_E_OFFSET;
    }
    return BDLM_OK;
}

int bdlm_check_commit(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                      const void *B, const void *C, const float *D, const float *D_rev,
                      const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                      const int64_t *n_committed, const int64_t *n_blocks,
                      int64_t expected_block_index) {
    int rc = check_common(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx,
                          BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    rc = check_long_block(d);
    if (rc != BDLM_OK) return rc;
    return check_books(d, slot_idx, n_committed, n_blocks, expected_block_index);
}

static int check_workspace(const void *ws, int64_t ws_bytes, int64_t need) {
    if (ws_bytes < 0) return BDLM_E_SHAPE;
    if (need == 0) return BDLM_OK;
    if (!ws) return BDLM_E_WORKSPACE;
    if (ws_bytes < need) return BDLM_E_WORKSPACE;
    if (!aligned(ws, 256)) return BDLM_E_ALIGN;
    return BDLM_OK;
}

int bdlm_full_window_workspace(const bdlm_desc_t *d, int64_t *bytes) {
    if (!bytes) return BDLM_E_NULL;
    const int rc = check_desc(d, BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    *bytes = bdlm::full_window_workspace(d->batch, d->nheads, d->dstate, d->block_len);
    return BDLM_OK;
}

int bdlm_prefill_workspace(const bdlm_desc_t *d, int64_t *bytes) {
    if (!bytes) return BDLM_E_NULL;
    const int rc = check_desc(d, BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    *bytes = bdlm::prefill_workspace(d->batch, d->nheads, d->dstate, d->block_len);
    return BDLM_OK;
}

int bdlm_check_full_window(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                           const void *B, const void *C, const float *D, const float *D_rev,
                           const float *y, const void *workspace, int64_t workspace_bytes) {
    int rc = check_common(d, x, dt, A, B, C, D, D_rev, nullptr, 0, nullptr, BDLM_MAX_SEQ_LEN,
                          false);
    if (rc != BDLM_OK) return rc;
    rc = check_seq_strides(d);
    if (rc != BDLM_OK) return rc;
    if (!y && d->batch != 0 && d->block_len != 0) return BDLM_E_NULL;
    if (!aligned(y, 4)) return BDLM_E_ALIGN;
    return check_workspace(workspace, workspace_bytes,
                           bdlm::full_window_workspace(d->batch, d->nheads, d->dstate,
                                                       d->block_len));
}

int bdlm_check_prefill(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                       const void *B, const void *C, const float *D, const float *h_pool,
                       int64_t nslots, const int32_t *slot_idx, const int64_t *n_committed,
                       const int64_t *n_blocks, int64_t expected_block_index,
                       int64_t blocks_in_prefix, const float *y_fwd, const void *workspace,
                       int64_t workspace_bytes) {
    // D_rev is not used by a forward-only pass; D stands in for it in the checks
    int rc = check_common(d, x, dt, A, B, C, D, D, h_pool, nslots, slot_idx, BDLM_MAX_SEQ_LEN,
                          true);
    if (rc != BDLM_OK) return rc;
    rc = check_seq_strides(d);
    if (rc != BDLM_OK) return rc;
    if (blocks_in_prefix < 0) return BDLM_E_SHAPE;
    if (!aligned(y_fwd, 4)) return BDLM_E_ALIGN;
    rc = check_workspace(workspace, workspace_bytes,
                         bdlm::prefill_workspace(d->batch, d->nheads, d->dstate, d->block_len));
    if (rc != BDLM_OK) return rc;
    return check_books(d, slot_idx, n_committed, n_blocks, expected_block_index);
}

int bdlm_boundary_states_workspace(const bdlm_desc_t *d, int64_t n_blocks, int64_t *bytes) {
    if (!bytes) return BDLM_E_NULL;
    const int rc = check_desc(d, BDLM_MAX_BLOCK_LEN);
    if (rc != BDLM_OK) return rc;
    if (n_blocks < 0) return BDLM_E_SHAPE;
    *bytes = bdlm::boundary_workspace(d->batch, d->nheads, d->dstate, n_blocks, d->block_len);
    return BDLM_OK;
}

int bdlm_check_block_boundary_states(const bdlm_desc_t *d, int64_t n_blocks, const void *x,
                                     const void *dt, const float *A, const void *B,
                                     const void *C, const float *D, const float *s_init,
                                     const float *s_out, const float *y_fwd,
                                     const void *workspace, int64_t workspace_bytes) {
    // the whole clean sequence is n_blocks * block_len tokens; check it as such
    if (!d) return BDLM_E_NULL;
    if (n_blocks < 0) return BDLM_E_SHAPE;
    if (d->block_len > BDLM_MAX_BLOCK_LEN || d->block_len < 0) return BDLM_E_SHAPE;
    if (d->block_len > 0 && n_blocks > BDLM_MAX_SEQ_LEN / d->block_len) return BDLM_E_SHAPE;
    bdlm_desc_t seq = *d;
    seq.block_len = d->block_len * n_blocks;
    // C is read only for the forward outputs
    int rc = check_common(&seq, x, dt, A, B, y_fwd ? C : B, D, D, nullptr, 0, nullptr,
                          BDLM_MAX_SEQ_LEN, false);
    if (rc != BDLM_OK) return rc;
    rc = check_seq_strides(&seq);
    if (rc != BDLM_OK) return rc;
    if (d->batch * d->nheads * n_blocks > (int64_t(1) << 30)) return BDLM_E_SHAPE;
    const bool empty = d->batch == 0 || seq.block_len == 0;
    if (!s_out && !empty) return BDLM_E_NULL;
    if (!aligned(s_out, 16) || !aligned(s_init, 16) || !aligned(y_fwd, 4)) return BDLM_E_ALIGN;
    return check_workspace(workspace, workspace_bytes,
                           empty ? 0
                                 : bdlm::boundary_workspace(d->batch, d->nheads, d->dstate,
                                                            n_blocks, d->block_len));
}

int bdlm_block_boundary_states(const bdlm_desc_t *d, int64_t n_blocks, const void *x,
                               const void *dt, const float *A, const void *B, const void *C,
                               const float *D, const float *s_init, float *s_out, float *y_fwd,
                               void *workspace, int64_t workspace_bytes, void *stream) {
    const int rc = bdlm_check_block_boundary_states(d, n_blocks, x, dt, A, B, C, D, s_init, s_out,
                                                    y_fwd, workspace, workspace_bytes);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs a = make_args(d, x, dt, A, B, C, D, D, nullptr, nullptr, y_fwd);
    return bdlm::launch_boundary_states(a, n_blocks, s_init, s_out, workspace, stream);
}

int bdlm_scan_block_step(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                         const void *B, const void *C, const float *D, const float *D_rev,
                         const float *h_pool, int64_t nslots, const int32_t *slot_idx, float *y,
                         void *stream) {
    const int rc =
        bdlm_check_block_step(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx, y);
    if (rc != BDLM_OK) return rc;
    // The step never writes the cache; the kernel receives it through the same
    // argument block as a commit, with the state update compiled out.
    const bdlm::LaunchArgs a =
        make_args(d, x, dt, A, B, C, D, D_rev, const_cast<float *>(h_pool), slot_idx, y);
    return by_row_chunks(a, y_row_floats(d, d->block_len), [&](const bdlm::LaunchArgs &c) {
        return d->block_len > BDLM_MAX_BLOCK_LEN ? bdlm::launch_block_long_shared(c, false, true, stream)
                                                 : bdlm::launch_block(c, false, stream);
    });
}

int bdlm_check_block_step_sep(const bdlm_desc_t *d, const void *x, const void *dt,
                              const float *A, const void *B, const void *C, const float *D,
                              const void *x_rev, const void *dt_rev, const float *A_rev,
                              const void *B_rev, const void *C_rev, const float *D_rev,
                              const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                              const float *y) {
    int rc = check_common(d, x, dt, A, B, C, D, D, h_pool, nslots, slot_idx, BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    rc = check_common(d, x_rev, dt_rev, A_rev, B_rev, C_rev, D_rev, D_rev, nullptr, 0, nullptr,
                      BDLM_MAX_SEQ_LEN, false);
    if (rc != BDLM_OK) return rc;
    rc = check_seq_strides(d);
    if (rc != BDLM_OK) return rc;
    if (!y && d->batch != 0 && d->block_len != 0) return BDLM_E_NULL;
    if (!aligned(y, 4)) return BDLM_E_ALIGN;
    return BDLM_OK;
}

int bdlm_scan_block_step_sep(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                             const void *B, const void *C, const float *D, const void *x_rev,
                             const void *dt_rev, const float *A_rev, const void *B_rev,
                             const void *C_rev, const float *D_rev, const float *h_pool,
                             int64_t nslots, const int32_t *slot_idx, float *y, void *stream) {
    const int rc = bdlm_check_block_step_sep(d, x, dt, A, B, C, D, x_rev, dt_rev, A_rev, B_rev,
                                             C_rev, D_rev, h_pool, nslots, slot_idx, y);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs f =
        make_args(d, x, dt, A, B, C, D, D, const_cast<float *>(h_pool), slot_idx, y);
    const bdlm::LaunchArgs r =
        make_args(d, x_rev, dt_rev, A_rev, B_rev, C_rev, D_rev, D_rev, nullptr, slot_idx, y);
    const int64_t yr = y_row_floats(d, d->block_len);
    return by_row_chunks(f, yr, [&](const bdlm::LaunchArgs &fc) {
        const int64_t r0 = fc.slots ? fc.slots - f.slots : 0;
        const bdlm::LaunchArgs rc = rows_of(r, r0, fc.batch, yr);
        return d->block_len <= BDLM_MAX_BLOCK_LEN ? bdlm::launch_block_pair(fc, rc, false, true, stream)
                                                  : bdlm::launch_block_long(fc, rc, false, true, stream);
    });
}

int bdlm_commit_boundary(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                         const void *B, const void *C, const float *D, const float *D_rev,
                         float *h_pool, int64_t nslots, const int32_t *slot_idx,
                         int64_t *n_committed, int64_t *n_blocks, int64_t expected_block_index,
                         float *y_clean, void *stream) {
    int rc = bdlm_check_commit(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx, n_committed,
                               n_blocks, expected_block_index);
    if (rc != BDLM_OK) return rc;
    if (y_clean && !aligned(y_clean, 16)) return BDLM_E_ALIGN;
    const bdlm::LaunchArgs a =
        make_args(d, x, dt, A, B, C, D, D_rev, h_pool, slot_idx, y_clean);
    rc = by_row_chunks(a, y_row_floats(d, d->block_len), [&](const bdlm::LaunchArgs &c) {
        return d->block_len > BDLM_MAX_BLOCK_LEN
                   ? bdlm::launch_block_long_shared(c, true, y_clean != nullptr, stream)
                   : bdlm::launch_block(c, true, stream);
    });
    if (rc != BDLM_OK) return rc;
    for (int64_t b = 0; b < d->batch; ++b) {
        const int64_t s = slot_idx ? slot_idx[b] : b;
        n_committed[s] += d->block_len;
        n_blocks[s] += 1;
    }
    return BDLM_OK;
}

int bdlm_check_commit_step(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                           const void *B, const void *C, const float *D, const float *D_rev,
                           const void *x_next, const void *dt_next, const void *B_next,
                           const void *C_next, const float *h_pool, int64_t nslots,
                           const int32_t *slot_idx, const int64_t *n_committed,
                           const int64_t *n_blocks, int64_t expected_block_index,
                           const float *y_clean, const float *y_next) {
    int rc = check_common(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx);
    if (rc != BDLM_OK) return rc;
    rc = check_common(d, x_next, dt_next, A, B_next, C_next, D, D_rev, nullptr, 0, nullptr,
                      BDLM_MAX_BLOCK_LEN, false);
    if (rc != BDLM_OK) return rc;
    if (!y_next && d->batch != 0 && d->block_len != 0) return BDLM_E_NULL;
    if (!aligned(y_next, 16) || !aligned(y_clean, 16)) return BDLM_E_ALIGN;
    return check_books(d, slot_idx, n_committed, n_blocks, expected_block_index);
}

int bdlm_commit_step(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                     const void *B, const void *C, const float *D, const float *D_rev,
                     const void *x_next, const void *dt_next, const void *B_next,
                     const void *C_next, float *h_pool, int64_t nslots, const int32_t *slot_idx,
                     int64_t *n_committed, int64_t *n_blocks, int64_t expected_block_index,
                     float *y_clean, float *y_next, void *stream) {
    int rc = bdlm_check_commit_step(d, x, dt, A, B, C, D, D_rev, x_next, dt_next, B_next, C_next,
                                    h_pool, nslots, slot_idx, n_committed, n_blocks,
                                    expected_block_index, y_clean, y_next);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs a = make_args(d, x, dt, A, B, C, D, D_rev, h_pool, slot_idx, y_clean);
    const bdlm::LaunchArgs n =
        make_args(d, x_next, dt_next, A, B_next, C_next, D, D_rev, h_pool, slot_idx, y_next);
    const int64_t yr = y_row_floats(d, d->block_len);
    rc = by_row_chunks(a, yr, [&](const bdlm::LaunchArgs &ac) -> int {
        const int64_t r0 = ac.slots ? ac.slots - a.slots : 0;
        const bdlm::LaunchArgs nc = rows_of(n, r0, ac.batch, yr);
        return bdlm::launch_commit_step(ac, nc, nc.y, stream);
    });
    if (rc != BDLM_OK) return rc;
    for (int64_t b = 0; b < d->batch; ++b) {
        const int64_t s = slot_idx ? slot_idx[b] : b;
        n_committed[s] += d->block_len;
        n_blocks[s] += 1;
    }
    return BDLM_OK;
}

int bdlm_conv_workspace(const bdlm_desc_t *d, int64_t *bytes) {
    if (!bytes) return BDLM_E_NULL;
    const int rc = check_desc(d, BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    *bytes = bdlm::conv_workspace(d->batch, d->block_len, d->nheads, d->ngroups, d->dstate);
    return BDLM_OK;
}

static int check_conv(const bdlm_desc_t *d, const float *conv_w, const float *conv_b,
                      const float *conv_pool, const void *ws, int64_t ws_bytes) {
    if (!conv_w || !conv_b || !conv_pool) return BDLM_E_NULL;
    // the kernels read weights, biases and cached rows as 16-byte vectors
    if (!aligned(conv_w, 16) || !aligned(conv_b, 16) || !aligned(conv_pool, 16)) return BDLM_E_ALIGN;
    // the convolved inputs are scanned from the (fp32, contiguous) workspace
    if (d->nheads * BDLM_HEADDIM * 4 > (int64_t(1) << 24)) return BDLM_E_SHAPE;
    return check_workspace(ws, ws_bytes,
                           bdlm::conv_workspace(d->batch, d->block_len, d->nheads, d->ngroups,
                                                d->dstate));
}

int bdlm_check_conv_block_step(const bdlm_desc_t *d, const void *x, const void *dt,
                               const float *A, const void *B, const void *C, const float *D,
                               const float *D_rev, const float *conv_w, const float *conv_b,
                               const float *conv_pool, const float *h_pool, int64_t nslots,
                               const int32_t *slot_idx, const float *y, const void *workspace,
                               int64_t workspace_bytes) {
    int rc = check_common(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx, BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    if (!y && d->batch != 0 && d->block_len != 0) return BDLM_E_NULL;
    if (!aligned(y, 4)) return BDLM_E_ALIGN;
    return check_conv(d, conv_w, conv_b, conv_pool, workspace, workspace_bytes);
}

int bdlm_conv_block_step(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                         const void *B, const void *C, const float *D, const float *D_rev,
                         const float *conv_w, const float *conv_b, const float *conv_pool,
                         const float *h_pool, int64_t nslots, const int32_t *slot_idx, float *y,
                         void *workspace, int64_t workspace_bytes, void *stream) {
    const int rc = bdlm_check_conv_block_step(d, x, dt, A, B, C, D, D_rev, conv_w, conv_b,
                                              conv_pool, h_pool, nslots, slot_idx, y, workspace,
                                              workspace_bytes);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs a =
        make_args(d, x, dt, A, B, C, D, D_rev, const_cast<float *>(h_pool), slot_idx, y);
    return by_row_chunks(a, y_row_floats(d, d->block_len), [&](const bdlm::LaunchArgs &c) {
        return bdlm::launch_conv_block(c, conv_w, conv_b, const_cast<float *>(conv_pool), false,
                                       workspace, stream);
    });
}

int bdlm_check_conv_commit(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                           const void *B, const void *C, const float *D, const float *D_rev,
                           const float *conv_w, const float *conv_b, const float *conv_pool,
                           const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                           const int64_t *n_committed, const int64_t *n_blocks,
                           int64_t expected_block_index, const float *y_clean,
                           const void *workspace, int64_t workspace_bytes) {
    int rc = check_common(d, x, dt, A, B, C, D, D_rev, h_pool, nslots, slot_idx, BDLM_MAX_SEQ_LEN);
    if (rc != BDLM_OK) return rc;
    if (!aligned(y_clean, 4)) return BDLM_E_ALIGN;
    rc = check_conv(d, conv_w, conv_b, conv_pool, workspace, workspace_bytes);
    if (rc != BDLM_OK) return rc;
    return check_books(d, slot_idx, n_committed, n_blocks, expected_block_index);
}

int bdlm_conv_commit_boundary(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                              const void *B, const void *C, const float *D, const float *D_rev,
                              const float *conv_w, const float *conv_b, float *conv_pool,
                              float *h_pool, int64_t nslots, const int32_t *slot_idx,
                              int64_t *n_committed, int64_t *n_blocks,
                              int64_t expected_block_index, float *y_clean, void *workspace,
                              int64_t workspace_bytes, void *stream) {
    int rc = bdlm_check_conv_commit(d, x, dt, A, B, C, D, D_rev, conv_w, conv_b, conv_pool, h_pool,
                                    nslots, slot_idx, n_committed, n_blocks, expected_block_index,
                                    y_clean, workspace, workspace_bytes);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs a = make_args(d, x, dt, A, B, C, D, D_rev, h_pool, slot_idx, y_clean);
    rc = by_row_chunks(a, y_row_floats(d, d->block_len), [&](const bdlm::LaunchArgs &c) {
        return bdlm::launch_conv_block(c, conv_w, conv_b, conv_pool, true, workspace, stream);
    });
    if (rc != BDLM_OK) return rc;
    for (int64_t b = 0; b < d->batch; ++b) {
        const int64_t s = slot_idx ? slot_idx[b] : b;
        n_committed[s] += d->block_len;
        n_blocks[s] += 1;
    }
    return BDLM_OK;
}

int bdlm_scan_full_window(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                          const void *B, const void *C, const float *D, const float *D_rev,
                          float *y, void *workspace, int64_t workspace_bytes, void *stream) {
    const int rc =
        bdlm_check_full_window(d, x, dt, A, B, C, D, D_rev, y, workspace, workspace_bytes);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs a = make_args(d, x, dt, A, B, C, D, D_rev, nullptr, nullptr, y);
    return bdlm::launch_full_window(a, d->block_len, workspace, stream);
}

int bdlm_prefill(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                 const void *B, const void *C, const float *D, float *h_pool, int64_t nslots,
                 const int32_t *slot_idx, int64_t *n_committed, int64_t *n_blocks,
                 int64_t expected_block_index, int64_t blocks_in_prefix, float *y_fwd,
                 void *workspace, int64_t workspace_bytes, void *stream) {
    int rc = bdlm_check_prefill(d, x, dt, A, B, C, D, h_pool, nslots, slot_idx, n_committed,
                                n_blocks, expected_block_index, blocks_in_prefix, y_fwd,
                                workspace, workspace_bytes);
    if (rc != BDLM_OK) return rc;
    const bdlm::LaunchArgs a = make_args(d, x, dt, A, B, C, D, D, h_pool, slot_idx, y_fwd);
    rc = by_row_chunks(a, y_row_floats(d, d->block_len), [&](const bdlm::LaunchArgs &c) {
        return bdlm::launch_prefill(c, d->block_len, workspace, stream);
    });
    if (rc != BDLM_OK) return rc;
    for (int64_t b = 0; b < d->batch; ++b) {
        const int64_t s = slot_idx ? slot_idx[b] : b;
        n_committed[s] += d->block_len;
        n_blocks[s] += blocks_in_prefix;
    }
    return BDLM_OK;
}

int bdlm_prefill_noalloc(const bdlm_desc_t *d, const void *x, const void *dt, const float *A,
                         const void *B, const void *C, const float *D, float *h_pool,
                         int64_t nslots, const int32_t *slot_idx, int64_t *n_committed,
                         int64_t *n_blocks, int64_t expected_block_index,
                         int64_t blocks_in_prefix, float *y_fwd, void *stream) {
    // the checks of bdlm_prefill with the workspace test replaced by the scratch plan
    void *const any = reinterpret_cast<void *>(uintptr_t(256));
    int rc = bdlm_check_prefill(d, x, dt, A, B, C, D, h_pool, nslots, slot_idx, n_committed,
                                n_blocks, expected_block_index, blocks_in_prefix, y_fwd, any,
                                INT64_MAX);
    if (rc != BDLM_OK) return rc;
    const int64_t rows = slot_idx && d->batch > BDLM_MAX_SLOT_ROWS ? BDLM_MAX_SLOT_ROWS : d->batch;
    bdlm::SeqPlan plan;
    if (d->batch > 0 && d->block_len > 0 &&
        !bdlm::prefill_plan_capped(rows, d->nheads, d->dstate, d->block_len, BDLM_SCRATCH_BYTES,
                                   &plan))
        return BDLM_E_WORKSPACE;
    void *ws = nullptr;
    if (d->batch > 0 && d->block_len > 0) {
        rc = bdlm::scratch_pointer(&ws);
        if (rc != BDLM_OK) return rc;
    }
    const bdlm::LaunchArgs a = make_args(d, x, dt, A, B, C, D, D, h_pool, slot_idx, y_fwd);
    rc = by_row_chunks(a, y_row_floats(d, d->block_len), [&](const bdlm::LaunchArgs &c) -> int {
        if (c.batch == 0 || d->block_len == 0) return BDLM_OK;   // nothing to enqueue
        bdlm::SeqPlan p;
        // a shorter last run of rows fits whenever a full one does
        if (!bdlm::prefill_plan_capped(c.batch, d->nheads, d->dstate, d->block_len,
                                       BDLM_SCRATCH_BYTES, &p))
            return BDLM_E_WORKSPACE;
        return bdlm::launch_prefill(c, d->block_len, ws, stream, &p);
    });
    if (rc != BDLM_OK) return rc;
    for (int64_t b = 0; b < d->batch; ++b) {
        const int64_t s = slot_idx ? slot_idx[b] : b;
        n_committed[s] += d->block_len;
        n_blocks[s] += blocks_in_prefix;
    }
    return BDLM_OK;
}

static int state_permute(const float *src, float *dst, int64_t nstates, int64_t dstate,
                         bool to_pool, void *stream) {
    if (!src || !dst) return BDLM_E_NULL;
    if (nstates < 0 || (dstate != 16 && dstate != 32 && dstate != 64 && dstate != 128))
        return BDLM_E_SHAPE;
    if (!aligned(src, 16) || !aligned(dst, 16)) return BDLM_E_ALIGN;
    const int64_t bytes = nstates * BDLM_HEADDIM * dstate * 4;
    const char *s = reinterpret_cast<const char *>(src), *t = reinterpret_cast<const char *>(dst);
    if (s < t + bytes && t < s + bytes && nstates > 0) return BDLM_E_SHAPE;  // overlap
    return bdlm::launch_state_permute(src, dst, nstates, dstate, to_pool, stream);
}

int bdlm_state_pack(const float *rowmajor, float *pool, int64_t nstates, int64_t dstate,
                    void *stream) {
    return state_permute(rowmajor, pool, nstates, dstate, true, stream);
}

int bdlm_state_unpack(const float *pool, float *rowmajor, int64_t nstates, int64_t dstate,
                      void *stream) {
    return state_permute(pool, rowmajor, nstates, dstate, false, stream);
}

int bdlm_cache_reset(float *h_pool, int64_t nslots, int64_t state_elems, const int32_t *slots,
                     int64_t nreset, int64_t *n_committed, int64_t *n_blocks, void *stream) {
    if (!h_pool) return BDLM_E_NULL;
    if (nslots <= 0 || state_elems <= 0 || state_elems % 4 != 0 || nreset < 0) return BDLM_E_SHAPE;
    if (!aligned(h_pool, 16)) return BDLM_E_ALIGN;
    if (slots)
        for (int64_t i = 0; i < nreset; ++i)
            if (slots[i] < 0 || slots[i] >= nslots) return BDLM_E_SLOT;
    const int rc = bdlm::launch_reset(h_pool, nslots, state_elems, slots, nreset, stream);
    if (rc != BDLM_OK) return rc;
    const int64_t count = slots ? nreset : nslots;
    for (int64_t i = 0; i < count; ++i) {
        const int64_t s = slots ? slots[i] : i;
        if (n_committed) n_committed[s] = 0;
        if (n_blocks) n_blocks[s] = 0;
    }
    return BDLM_OK;
}

namespace {
bool disjoint(const void *a, int64_t abytes, const void *b, int64_t bbytes) {
    const char *p = static_cast<const char *>(a), *q = static_cast<const char *>(b);
    return abytes <= 0 || bbytes <= 0 || p + abytes <= q || q + bbytes <= p;
}
}  // namespace

int bdlm_check_gated_rmsnorm(int64_t batch, int64_t len, int64_t nheads, int64_t ngroups,
                             int32_t z_dtype, const float *y, const void *z, int64_t z_stride_b,
                             int64_t z_stride_t, const float *norm_w, float eps,
                             const float *out) {
    if (z_dtype != BDLM_DTYPE_F32 && z_dtype != BDLM_DTYPE_BF16) return BDLM_E_DTYPE;
    if (batch < 0 || len < 0 || nheads <= 0 || nheads > BDLM_NORM_MAX_HEADS || ngroups <= 0 ||
        nheads % ngroups != 0)
        return BDLM_E_SHAPE;
    if (z_stride_b < 0 || z_stride_t < 0) return BDLM_E_SHAPE;
    if (!(eps >= 0.f && eps <= 3.0e38f)) return BDLM_E_SHAPE;   // finite, not negative, not NaN
    constexpr int64_t kMax = int64_t(1) << 31;
    if (batch > kMax || len > kMax || (len > 0 && batch > (int64_t(1) << 40) / len))
        return BDLM_E_SHAPE;
    if (!norm_w) return BDLM_E_NULL;
    const bool empty = batch == 0 || len == 0;
    if (!empty && (!y || !z || !out)) return BDLM_E_NULL;
    const int64_t es = elem_size(z_dtype);
    if (!aligned(y, 16) || !aligned(out, 16) || !aligned(norm_w, 16) || !aligned(z, 4 * es))
        return BDLM_E_ALIGN;
    if (z_stride_b % 4 != 0 || z_stride_t % 4 != 0) return BDLM_E_ALIGN;
    if (empty) return BDLM_OK;
    const int64_t ch = nheads * BDLM_HEADDIM;
    if (z_stride_b > (int64_t(1) << 40) || z_stride_t > (int64_t(1) << 40)) return BDLM_E_SHAPE;
    const int64_t ybytes = batch * len * ch * 4;
    const int64_t zbytes = ((batch - 1) * z_stride_b + (len - 1) * z_stride_t + ch) * es;
    // out may be y itself (in place); no other overlap with an input
    if (out != y && !disjoint(out, ybytes, y, ybytes)) return BDLM_E_SHAPE;
    if (!disjoint(out, ybytes, z, zbytes) || !disjoint(out, ybytes, norm_w, ch * 4))
        return BDLM_E_SHAPE;
    return BDLM_OK;
}

int bdlm_gated_rmsnorm(int64_t batch, int64_t len, int64_t nheads, int64_t ngroups,
                       int32_t z_dtype, const float *y, const void *z, int64_t z_stride_b,
                       int64_t z_stride_t, const float *norm_w, float eps, float *out,
                       void *stream) {
    const int rc = bdlm_check_gated_rmsnorm(batch, len, nheads, ngroups, z_dtype, y, z,
                                            z_stride_b, z_stride_t, norm_w, eps, out);
    if (rc != BDLM_OK) return rc;
    bdlm::NormLaunch n;
    n.y = y;
    n.z = z;
    n.w = norm_w;
    n.out = out;
    n.zs_b = z_stride_b;
    n.zs_t = z_stride_t;
    n.batch = batch;
    n.len = len;
    n.nheads = nheads;
    n.ngroups = ngroups;
    n.bf16 = z_dtype == BDLM_DTYPE_BF16 ? 1 : 0;
    n.eps = eps;
    return bdlm::launch_gated_rmsnorm(n, stream);
}

}  // extern "C"
