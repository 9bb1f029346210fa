/*
 * bdlm.h -- C ABI of libbdlm: the block-restricted bidirectional Mamba scan of
 * BDLM Mamba-H on AMD Instinct MI355X (gfx950).
 *
 * Paper: "Training Hybrid Block Diffusion Language Models with Partial
 * Bidirectionality".  Per Mamba layer, the BDLM sampler keeps one forward
 * boundary state per sequence (Sec. 4, Eq. boundary-state).  Every denoising
 * step of the active block continues that state forward through the block,
 * runs a reverse scan of the block from a zero state, and sums the two outputs
 * (Sec. 4, Eq. partial-reverse).  Once the block is final, the clean block's
 * forward state replaces the cached one (the cache-append step of the BDLM
 * sampler, Sec. 3; Sec. 4.1).
 *
 * Recurrence (Sec. 3, Eq. mamba-scan-background, in the Mamba-2 form the
 * paper's mixers use, App. C).  For batch row b, head h, group g = h / (H/G):
 *     a_t = exp(dt[b,t,h] * A[h])
 *     S_t = a_t S_{t-1} + dt[b,t,h] * x[b,t,h,:] (outer) B[b,t,g,:]      (P x N)
 *     out_t = S_t C[b,t,g,:] + skip * x[b,t,h,:]
 * Forward branch: S_{-1} = cached state, skip = D[h].
 * Reverse branch: tokens in reversed order (each keeps its own x, dt, B, C),
 * S = 0 before the last token, skip = D_rev[h].   y = forward + reverse.
 *
 * Conventions shared by every entry point:
 *   - Device pointers point to device memory the caller allocated and owns.
 *     The library never allocates, frees or synchronises, and keeps no pointer
 *     after returning.  Work is enqueued on `stream` (a hipStream_t; NULL is the
 *     null stream) and runs asynchronously.
 *   - Host pointers (slot_idx, n_committed, n_blocks) are read, and for a commit
 *     updated, before the call returns.
 *   - Every check happens on the host before anything is enqueued; on any
 *     error nothing is enqueued and nothing is modified.  The return value is
 *     BDLM_OK or a negative BDLM_E_* code.  No entry point aborts.
 *   - Sizes: headdim P == 64; dstate N in {16, 32, 64, 128}; block_len L in
 *     [0, BDLM_MAX_SEQ_LEN]; nheads % ngroups == 0; batch >= 0; batch * nheads
 *     <= 2^22 (within the 32-bit grid of a launch).  A block step or commit with
 *     L <= BDLM_MAX_BLOCK_LEN is one fused launch; longer blocks need per-token
 *     strides (and nheads * 64 * 4) of at most 16 MiB and run, with bf16 activations
 *     and L <= 256 (the paper's block length), as one launch computing the whole block
 *     in masked-matrix form, else on the sequence kernels as a forward launch from the
 *     cached state and a reverse launch adding into y.
 *   - Activation storage (x, dt, B, C) is fp32 or bf16 (desc.in_dtype).  All
 *     arithmetic, states and outputs are fp32.
 */
#ifndef BDLM_H
#define BDLM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BDLM_ABI_VERSION 1
#define BDLM_HEADDIM 64
#define BDLM_MAX_BLOCK_LEN 64
/* Longest sequence of bdlm_scan_full_window and bdlm_prefill. */
#define BDLM_MAX_SEQ_LEN (((int64_t)1 << 31) - 1)
/* Rows per launch when an explicit slot_idx is given: the kernels receive the slot
   table by value, so a call with a longer table is enqueued as consecutive launches of
   at most this many rows (no limit on batch results from it). */
#define BDLM_MAX_SLOT_ROWS 256
/* Most heads (nheads * 64 channels) bdlm_gated_rmsnorm takes per token. */
#define BDLM_NORM_MAX_HEADS 256

enum bdlm_status {
    BDLM_OK = 0,
    BDLM_E_NULL = -1,    /* a required pointer is NULL */
    BDLM_E_SHAPE = -2,   /* a size is unsupported or inconsistent */
    BDLM_E_DTYPE = -3,   /* unknown in_dtype, or reserved field not zero */
    BDLM_E_ALIGN = -4,   /* a pointer or stride breaks the alignment contract */
    BDLM_E_OFFSET = -5,  /* commit: a slot does not hold expected_block_index blocks */
    BDLM_E_SLOT = -6,    /* slot index out of range, or repeated within one commit */
    BDLM_E_LAUNCH = -7,  /* the HIP runtime refused the launch */
    BDLM_E_WORKSPACE = -8 /* sequence entry points: workspace missing or too small */
};

enum bdlm_dtype { BDLM_DTYPE_F32 = 0, BDLM_DTYPE_BF16 = 1 };

/*
 * Shape and activation layout of one call.  Strides are in elements.
 *   x  [batch][block_len][nheads][headdim]: x_stride = {batch, token, head};
 *      headdim is unit stride.
 *   dt [batch][block_len][nheads]: dt_stride = {batch, token}; heads unit stride.
 *   B, C [batch][block_len][ngroups][dstate]: bc_stride = {batch, token, group};
 *      dstate unit stride; B and C share strides.
 * Strides may describe views into a larger projection output (e.g. slices of a
 * Mamba-2 in_proj result).  bdlm_desc_init fills contiguous strides.
 */
typedef struct bdlm_desc {
    int64_t batch;
    int64_t nheads;
    int64_t headdim;
    int64_t dstate;
    int64_t ngroups;
    int64_t block_len;
    int32_t in_dtype;   /* enum bdlm_dtype */
    int32_t reserved;   /* must be 0 */
    int64_t x_stride[3];
    int64_t dt_stride[2];
    int64_t bc_stride[3];
} bdlm_desc_t;

/* Version of this ABI (BDLM_ABI_VERSION). */
int bdlm_abi_version(void);

/* Static, NUL-terminated description of a status code; never NULL. */
const char *bdlm_strerror(int status);

/* Fill *desc for contiguous activations.  Returns BDLM_E_NULL if desc is NULL,
   else BDLM_OK (sizes are checked by the entry points, not here). */
int bdlm_desc_init(bdlm_desc_t *desc, int64_t batch, int64_t nheads, int64_t headdim,
                   int64_t dstate, int64_t ngroups, int64_t block_len, int32_t in_dtype);

/*
 * Active-block denoising step (Sec. 4, Eq. partial-reverse).
 *
 *   y[b,t,h,:] = forward branch from the state h_pool[slot(b), h]
 *              + reverse branch of the block from zero
 *
 * x, dt, B, C  device, layout per desc, in_dtype storage.  Only the L block
 *              tokens are passed, so the reverse branch cannot see anything
 *              outside the block and the prefix enters only through h_pool.
 * A, D, D_rev  device fp32 [nheads].  A[h] < 0 keeps every decay below 1.
 * h_pool       device fp32 state pool, nslots x nheads states of 64 x dstate,
 *              16-byte aligned, in the pool layout (see bdlm_state_pack).  Read
 *              only (the cache is never written by a step).
 * slot_idx     host int32 array of exactly batch entries mapping batch row -> cache
 *              slot (entry b is row b's slot; the library reads entries 0 .. batch-1
 *              and nothing beyond), or NULL for slot(b) = b.  With more than
 *              BDLM_MAX_SLOT_ROWS rows the step is enqueued as one launch per run
 *              of that many rows.  Rows may share a slot.
 * y            device fp32 [batch][block_len][nheads][64], contiguous, 16-byte
 *              aligned.  Fully overwritten.  Must not overlap any input.
 * Alignment: x, B and C base pointers 16-byte aligned, and every x_stride and
 * bc_stride entry a multiple of 16 bytes (8 bf16 or 4 fp32 elements); dt, A, D,
 * D_rev and y aligned to their element size.
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE, BDLM_E_DTYPE, BDLM_E_ALIGN, BDLM_E_SLOT,
 * BDLM_E_LAUNCH.  batch == 0 or block_len == 0 enqueues nothing; x, dt, B, C and
 * y may then be NULL.
 */
int bdlm_scan_block_step(const bdlm_desc_t *desc, const void *x, const void *dt,
                         const float *A, const void *B, const void *C, const float *D,
                         const float *D_rev, const float *h_pool, int64_t nslots,
                         const int32_t *slot_idx, float *y, void *stream);

/*
 * Block finalisation: commit the clean block's forward boundary state
 * (Sec. 4, Eq. boundary-state; cache append of Sec. 3 and Sec. 4.1).
 *
 *   h_pool[slot(b), h] <- forward state after the L clean tokens, continued
 *                          from h_pool[slot(b), h]
 *   n_committed[slot(b)] += L;  n_blocks[slot(b)] += 1
 *
 * Inputs as for bdlm_scan_block_step, but h_pool is updated in place and the
 * rows' slots must be distinct.
 * n_committed, n_blocks  host int64 [nslots]: tokens and blocks committed per
 *              slot.  Every row's slot must satisfy n_blocks[slot] ==
 *              expected_block_index (pass a negative value to skip the check).
 *              Updated only after the launch has been enqueued successfully.
 * y_clean      device fp32 [batch][block_len][nheads][64] (16-byte aligned) or NULL.  If given, it
 *              receives the layer output on the clean block, computed exactly as
 *              bdlm_scan_block_step would from the state before the update.
 * Errors: as bdlm_scan_block_step, plus BDLM_E_OFFSET, and BDLM_E_SLOT for a
 * repeated slot.  block_len == 0 leaves states unchanged but still counts a
 * block.
 */
int bdlm_commit_boundary(const bdlm_desc_t *desc, const void *x, const void *dt,
                         const float *A, const void *B, const void *C, const float *D,
                         const float *D_rev, float *h_pool, int64_t nslots,
                         const int32_t *slot_idx, int64_t *n_committed, int64_t *n_blocks,
                         int64_t expected_block_index, float *y_clean, void *stream);

/*
 * Commit of the clean block followed by the first denoising step of the next block, in
 * the order the sampler takes them, as one call: the same results as
 * bdlm_commit_boundary(clean block) and then bdlm_scan_block_step(next block's noised
 * inputs) on the same stream (Eq. boundary-state, then Eq. partial-reverse from the new
 * state).  For bf16 blocks of at most 32 tokens it is one launch that reads each cached
 * state once, updates it in registers, writes it and continues the next block's step
 * from it, saving the step's read of the state; otherwise the two launches are enqueued.
 * The paper runs the clean forward pass and the next block's steps as separate passes;
 * this entry point is an alternative ordering of the same computation, not a change of
 * its results.
 *
 * x, dt, B, C                      the clean block (as for bdlm_commit_boundary);
 * x_next, dt_next, B_next, C_next  the next block's noised inputs at its first step,
 *              with desc's shapes and strides (same block length, same slots);
 * A, D, D_rev  shared by both (one layer).
 * h_pool, nslots, slot_idx, n_committed, n_blocks, expected_block_index, y_clean
 *              as for bdlm_commit_boundary (slots distinct, bookkeeping advanced by one
 *              block on success).
 * y_next       device fp32 [batch][block_len][nheads][64], 16-byte aligned, required:
 *              the next block's step outputs, from the committed state.
 * Blocks of at most BDLM_MAX_BLOCK_LEN tokens.
 * Errors: as bdlm_commit_boundary, with the next block's inputs checked as a step's.
 */
int bdlm_commit_step(const bdlm_desc_t *desc, const void *x, const void *dt, const float *A,
                     const void *B, const void *C, const float *D, const float *D_rev,
                     const void *x_next, const void *dt_next, const void *B_next,
                     const void *C_next, float *h_pool, int64_t nslots, const int32_t *slot_idx,
                     int64_t *n_committed, int64_t *n_blocks, int64_t expected_block_index,
                     float *y_clean, float *y_next, void *stream);

/*
 * The sequence entry points below split the sequence into segments, one
 * workgroup per (batch row, head, segment), and carry states between segments
 * through a device workspace that the caller allocates (the library allocates
 * nothing).  These return in *bytes the workspace size that bdlm_scan_full_window /
 * bdlm_prefill need for *desc (desc.block_len = sequence length); 0 means none.
 * The size depends only on batch, nheads, dstate and the length.
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE, BDLM_E_DTYPE.
 */
int bdlm_full_window_workspace(const bdlm_desc_t *desc, int64_t *bytes);
int bdlm_prefill_workspace(const bdlm_desc_t *desc, int64_t *bytes);

/*
 * One denoising step with separate reverse-direction inputs (Eq. partial-reverse with
 * F_theta,<- carrying its own projections): the forward branch runs on (x, dt, A, B,
 * C) from the cached state with skip D, the reverse branch on (x_rev, dt_rev, A_rev,
 * B_rev, C_rev) from zero with skip D_rev, and y is their sum.  Both input sets share
 * desc's shapes and strides; everything else as bdlm_scan_block_step (any block
 * length; bf16 blocks of up to 32 tokens in one launch, otherwise two: forward, then
 * reverse adding into y).
 * Errors: as bdlm_scan_block_step.
 */
int bdlm_scan_block_step_sep(const bdlm_desc_t *desc, const void *x, const void *dt,
                             const float *A, const void *B, const void *C, const float *D,
                             const void *x_rev, const void *dt_rev, const float *A_rev,
                             const void *B_rev, const void *C_rev, const float *D_rev,
                             const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                             float *y, void *stream);

/*
 * Block step and commit with the convolution part of the Mamba boundary state
 * (Sec. 2 and Sec. 4: the cached state includes the convolution state; App. C:
 * convolution width 4).  x, B and C are the block's inputs BEFORE the mixer's
 * depthwise causal convolution; per batch row b, channel c of xBC (x head-major
 * h * 64 + p, then B g * dstate + n, then C), with weights conv_w[c][0..3]
 * (conv_w[c][3] on the current token) and bias conv_b[c]:
 *   forward branch  xf[t] = silu(conv_b[c] + sum_k conv_w[c][k] u[t - 3 + k]), u[-3..-1]
 *                   the cached rows conv_pool[slot][0..2][c] (row 0 the oldest);
 *   reverse branch  xr[t] = silu(conv_b[c] + sum_k conv_w[c][k] u[t + 3 - k]), zero past
 *                   the block's end (the reverse branch stays inside the block);
 * then the step of bdlm_scan_block_step_sep with the forward branch on (xf, dt, A, Bf,
 * Cf, D) from the cached state and the reverse branch on (xr, dt, A, Br, Cr, D_rev)
 * from zero.  A commit also replaces the slot's conv_pool rows by the last three rows
 * of (cached rows ++ block) and updates h_pool from the forward branch.
 * conv_w       device fp32 [channels][4]; conv_b fp32 [channels].
 * conv_pool    device fp32 [nslots][3][channels] (same slots as h_pool).
 *              conv_w, conv_b and conv_pool are read as 16-byte vectors: all three
 *              must be 16-byte aligned (else BDLM_E_ALIGN).
 * workspace    at least bdlm_conv_workspace bytes (the convolved inputs, fp32),
 *              256-byte aligned; bf16 blocks of up to 32 tokens convolve inside
 *              the scan kernel's staging and leave it untouched.
 * Any block length.  Launches: a forward and a reverse scan launch, preceded by a
 * convolution launch into the workspace unless the block convolves in the staging;
 * a commit adds one launch that replaces the cached rows.  Errors: as
 * bdlm_scan_block_step / bdlm_commit_boundary, and BDLM_E_WORKSPACE.
 */
int bdlm_conv_workspace(const bdlm_desc_t *desc, int64_t *bytes);
int bdlm_conv_block_step(const bdlm_desc_t *desc, const void *x, const void *dt, const float *A,
                         const void *B, const void *C, const float *D, const float *D_rev,
                         const float *conv_w, const float *conv_b, const float *conv_pool,
                         const float *h_pool, int64_t nslots, const int32_t *slot_idx, float *y,
                         void *workspace, int64_t workspace_bytes, void *stream);
int bdlm_conv_commit_boundary(const bdlm_desc_t *desc, const void *x, const void *dt,
                              const float *A, const void *B, const void *C, const float *D,
                              const float *D_rev, const float *conv_w, const float *conv_b,
                              float *conv_pool, float *h_pool, int64_t nslots,
                              const int32_t *slot_idx, int64_t *n_committed, int64_t *n_blocks,
                              int64_t expected_block_index, float *y_clean, void *workspace,
                              int64_t workspace_bytes, void *stream);

/*
 * Full-window bidirectional scan, with no cache: the full-sequence
 * (DiffuMamba-style) scan that the paper's block-restricted scan replaces
 * (Sec. 4; Sec. 5.1).
 *
 *   y = forward scan over all desc.block_len tokens from a zero state (skip D)
 *     + reverse scan over all desc.block_len tokens from a zero state (skip D_rev)
 *
 * desc.block_len is the window length, 0 .. BDLM_MAX_SEQ_LEN; every other argument
 * is as for bdlm_scan_block_step with block_len set to the window (y is
 * [batch][window][nheads][64] fp32, 4-byte aligned).
 * Strides: every per-token stride (x, dt, B/C) and nheads * 64 * 4 (y's) at most
 * 16 MiB, else BDLM_E_SHAPE.
 * workspace    device memory of at least bdlm_full_window_workspace bytes,
 *              256-byte aligned (may be NULL when that size is 0); its contents
 *              are scratch, overwritten by the call.  Calls that share a
 *              workspace must not run concurrently.
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE, BDLM_E_DTYPE, BDLM_E_ALIGN,
 * BDLM_E_WORKSPACE, BDLM_E_LAUNCH.
 */
int bdlm_scan_full_window(const bdlm_desc_t *desc, const void *x, const void *dt,
                          const float *A, const void *B, const void *C, const float *D,
                          const float *D_rev, float *y, void *workspace,
                          int64_t workspace_bytes, void *stream);

/*
 * Chunked prefix prefill: summarise a clean prefix of desc.block_len tokens (any
 * length up to BDLM_MAX_SEQ_LEN) into the cached forward boundary states
 * (Eq. boundary-state), continuing each row's state in place.  Equivalent to
 * committing the prefix block by block.
 * h_pool, slot_idx  as for bdlm_commit_boundary (slots distinct).
 * n_committed, n_blocks  host bookkeeping: every slot must hold
 *              expected_block_index blocks (negative: unchecked); on success
 *              n_committed += desc.block_len and n_blocks += blocks_in_prefix
 *              (the number of sampler blocks the prefix spans, >= 0).
 * y_fwd        fp32 [batch][len][nheads][64] (4-byte aligned) or NULL: the forward
 *              outputs (skip D) of the prefix tokens.  D_rev is not used.
 * workspace    at least bdlm_prefill_workspace bytes, 256-byte aligned; scratch.
 * Strides as for bdlm_scan_full_window.
 * Errors: as bdlm_commit_boundary, and BDLM_E_WORKSPACE.
 */
int bdlm_prefill(const bdlm_desc_t *desc, const void *x, const void *dt, const float *A,
                 const void *B, const void *C, const float *D, float *h_pool, int64_t nslots,
                 const int32_t *slot_idx, int64_t *n_committed, int64_t *n_blocks,
                 int64_t expected_block_index, int64_t blocks_in_prefix, float *y_fwd,
                 void *workspace, int64_t workspace_bytes, void *stream);

/*
 * bdlm_prefill without a workspace argument, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Same arguments, semantics, bookkeeping and errors as bdlm_prefill; the
 * segment states live in a device array the library owns (BDLM_SCRATCH_BYTES per
 * device, held from the time the library's code is loaded on a device until the
 * process ends).  The call allocates nothing (no hipMalloc, no allocating library
 * routine).  When the standard segment plan needs more than BDLM_SCRATCH_BYTES it uses
 * fewer, longer segments; a call whose batch * nheads states do not fit even with one
 * segment (batch * nheads * 64 * dstate * 4 bytes above BDLM_SCRATCH_BYTES, per run of
 * BDLM_MAX_SLOT_ROWS rows when slot_idx is given) returns BDLM_E_WORKSPACE and
 * enqueues nothing.  Nothing in the scratch needs to start at zero: every value a call
 * reads was written by that call.  All calls on one device share its scratch, so calls
 * that may run concurrently on one device (on different streams) race; serialise them.
 */
#define BDLM_SCRATCH_BYTES ((int64_t)64 << 20)
int bdlm_prefill_noalloc(const bdlm_desc_t *desc, const void *x, const void *dt, const float *A,
                         const void *B, const void *C, const float *D, float *h_pool,
                         int64_t nslots, const int32_t *slot_idx, int64_t *n_committed,
                         int64_t *n_blocks, int64_t expected_block_index,
                         int64_t blocks_in_prefix, float *y_fwd, void *stream);

/*
 * All-block states of a clean sequence (the training computation of Fig. 1: every
 * block of a training window is denoised from the forward boundary state of its
 * clean prefix, Eq. prefix-cache-loss).  The clean sequence is n_blocks blocks of
 * desc.block_len (1 .. 64) tokens: x [batch][n_blocks * block_len][nheads][64] etc.
 * with desc's strides.
 * s_init       device fp32, batch x nheads states in the pool layout (the states
 *              before block 0), or NULL for zero states.
 * s_out        device fp32, batch * n_blocks * nheads states in the pool layout:
 *              state (row * n_blocks + k) * nheads + head is the forward state after
 *              blocks 0 .. k-1 of that row (k = 0: s_init).  16-byte aligned.
 * y_fwd        fp32 [batch][n_blocks * block_len][nheads][64] or NULL: the forward
 *              outputs (skip D) of the clean sequence.  C is read only for these.
 * workspace    at least bdlm_boundary_states_workspace bytes (one float per row,
 *              head and block), 256-byte aligned.
 * The noised blocks are then one bdlm_scan_block_step with batch batch * n_blocks
 * over s_out (slot_idx NULL): a contiguous [batch][n_blocks * block_len][...] tensor
 * is the same memory as [batch * n_blocks][block_len][...].
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE (also batch * nheads * n_blocks > 2^30),
 * BDLM_E_DTYPE, BDLM_E_ALIGN, BDLM_E_WORKSPACE, BDLM_E_LAUNCH.
 */
int bdlm_boundary_states_workspace(const bdlm_desc_t *desc, int64_t n_blocks, int64_t *bytes);
int bdlm_block_boundary_states(const bdlm_desc_t *desc, int64_t n_blocks, const void *x,
                               const void *dt, const float *A, const void *B, const void *C,
                               const float *D, const float *s_init, float *s_out, float *y_fwd,
                               void *workspace, int64_t workspace_bytes, void *stream);

/*
 * State pool layout.  The state of one (slot, head) is the 64 x dstate matrix
 * s[p][n] of the recurrence.  In a pool, state k = slot * nheads + head starts
 * at float offset k * 64 * dstate and stores s[p][n] at
 *     ((n / 4) * 64 + p) * 4 + n % 4,
 * i.e. dstate/4 blocks of [64][4]: groups of four consecutive state columns,
 * row by row.  The kernels read and write whole 16-byte groups, and a 64-wide
 * wave then moves 1 KB of contiguous memory per instruction.
 *
 * bdlm_state_pack copies nstates row-major states (s[p][n] at p * dstate + n)
 * into the pool layout; bdlm_state_unpack does the reverse.  Both pointers are
 * device fp32, 16-byte aligned, and must not overlap.
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE (dstate not in {16, 32, 64, 128}, nstates < 0,
 * or overlap), BDLM_E_ALIGN, BDLM_E_LAUNCH.
 */
int bdlm_state_pack(const float *rowmajor, float *pool, int64_t nstates, int64_t dstate,
                    void *stream);
int bdlm_state_unpack(const float *pool, float *rowmajor, int64_t nstates, int64_t dstate,
                      void *stream);

/*
 * Reset cache slots to the empty prefix: states to zero (with a fill kernel,
 * so the call is safe inside stream capture) and n_committed / n_blocks to 0.
 * h_pool       device fp32 [nslots][state_elems], 16-byte aligned.
 * slots        host int32 [nreset], each in [0, nslots); NULL resets all slots.
 * n_committed, n_blocks  host int64 [nslots], may both be NULL.
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE, BDLM_E_ALIGN, BDLM_E_SLOT, BDLM_E_LAUNCH.
 */
int bdlm_cache_reset(float *h_pool, int64_t nslots, int64_t state_elems, const int32_t *slots,
                     int64_t nreset, int64_t *n_committed, int64_t *n_blocks, void *stream);

/*
 * Gated RMS normalisation of the scan output, the step after the scan in the
 * Mamba-2 mixers the paper's Mamba layers use (App. C; the paper states no formula,
 * the Mamba-2 mixer's output path is taken):
 *
 *   g[c]   = y[c] * silu(z[c]),              silu(v) = v / (1 + exp(-v))
 *   out[c] = norm_w[c] * g[c] / sqrt(mean over c's group of g^2 + eps)
 *
 * per token (batch row, position), over the nheads * 64 channels (head-major, the
 * layout of y from every scan entry point), in ngroups groups of nheads / ngroups
 * whole heads.
 *
 * y        device fp32 [batch][len][nheads * 64], contiguous, 16-byte aligned.
 * z        device [batch][len][nheads * 64], z_dtype storage (BDLM_DTYPE_F32 or
 *          BDLM_DTYPE_BF16); element strides z_stride_b, z_stride_t (multiples of
 *          4, e.g. a slice of an in_proj output), unit channel stride; base aligned
 *          to 4 elements.
 * norm_w   device fp32 [nheads * 64], 16-byte aligned.
 * eps      finite, >= 0.
 * out      device fp32, y's layout, 16-byte aligned; may be y itself (in place);
 *          must not overlap z or norm_w, nor partly overlap y.
 * 1 <= nheads <= BDLM_NORM_MAX_HEADS; nheads % ngroups == 0.  batch == 0 or
 * len == 0 enqueues nothing (y, z and out may then be NULL).
 * Errors: BDLM_E_NULL, BDLM_E_SHAPE, BDLM_E_DTYPE, BDLM_E_ALIGN, BDLM_E_LAUNCH.
 */
int bdlm_gated_rmsnorm(int64_t batch, int64_t len, int64_t nheads, int64_t ngroups,
                       int32_t z_dtype, const float *y, const void *z, int64_t z_stride_b,
                       int64_t z_stride_t, const float *norm_w, float eps, float *out,
                       void *stream);

/*
 * Host-only argument checks used by the entry points above, exported so they
 * can be exercised without a GPU.  Same arguments (the stream is not needed),
 * same return codes; nothing is enqueued and nothing is modified.
 */
int bdlm_check_block_step(const bdlm_desc_t *desc, const void *x, const void *dt,
                          const float *A, const void *B, const void *C, const float *D,
                          const float *D_rev, const float *h_pool, int64_t nslots,
                          const int32_t *slot_idx, const float *y);
int bdlm_check_commit(const bdlm_desc_t *desc, const void *x, const void *dt, const float *A,
                      const void *B, const void *C, const float *D, const float *D_rev,
                      const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                      const int64_t *n_committed, const int64_t *n_blocks,
                      int64_t expected_block_index);
int bdlm_check_block_step_sep(const bdlm_desc_t *desc, const void *x, const void *dt,
                              const float *A, const void *B, const void *C, const float *D,
                              const void *x_rev, const void *dt_rev, const float *A_rev,
                              const void *B_rev, const void *C_rev, const float *D_rev,
                              const float *h_pool, int64_t nslots, const int32_t *slot_idx,
                              const float *y);
int bdlm_check_conv_block_step(const bdlm_desc_t *desc, const void *x, const void *dt,
                               const float *A, const void *B, const void *C, const float *D,
                               const float *D_rev, const float *conv_w, const float *conv_b,
                               const float *conv_pool, const float *h_pool, int64_t nslots,
                               const int32_t *slot_idx, const float *y, const void *workspace,
                               int64_t workspace_bytes);
int bdlm_check_conv_commit(const bdlm_desc_t *desc, const void *x, const void *dt,
                           const float *A, const void *B, const void *C, const float *D,
                           const float *D_rev, const float *conv_w, const float *conv_b,
                           const float *conv_pool, const float *h_pool, int64_t nslots,
                           const int32_t *slot_idx, const int64_t *n_committed,
                           const int64_t *n_blocks, int64_t expected_block_index,
                           const float *y_clean, const void *workspace, int64_t workspace_bytes);
int bdlm_check_commit_step(const bdlm_desc_t *desc, const void *x, const void *dt,
                           const float *A, const void *B, const void *C, const float *D,
                           const float *D_rev, const void *x_next, const void *dt_next,
                           const void *B_next, const void *C_next, const float *h_pool,
                           int64_t nslots, const int32_t *slot_idx, const int64_t *n_committed,
                           const int64_t *n_blocks, int64_t expected_block_index,
                           const float *y_clean, const float *y_next);
int bdlm_check_full_window(const bdlm_desc_t *desc, const void *x, const void *dt,
                           const float *A, const void *B, const void *C, const float *D,
                           const float *D_rev, const float *y, const void *workspace,
                           int64_t workspace_bytes);
int bdlm_check_block_boundary_states(const bdlm_desc_t *desc, int64_t n_blocks, const void *x,
                                     const void *dt, const float *A, const void *B,
                                     const void *C, const float *D, const float *s_init,
                                     const float *s_out, const float *y_fwd,
                                     const void *workspace, int64_t workspace_bytes);
int bdlm_check_gated_rmsnorm(int64_t batch, int64_t len, int64_t nheads, int64_t ngroups,
                             int32_t z_dtype, const float *y, const void *z, int64_t z_stride_b,
                             int64_t z_stride_t, const float *norm_w, float eps,
                             const float *out);
int bdlm_check_prefill(const bdlm_desc_t *desc, const void *x, const void *dt, const float *A,
                       const void *B, const void *C, const float *D, const float *h_pool,
                       int64_t nslots, const int32_t *slot_idx, const int64_t *n_committed,
                       const int64_t *n_blocks, int64_t expected_block_index,
                       int64_t blocks_in_prefix, const float *y_fwd, const void *workspace,
                       int64_t workspace_bytes);

#ifdef __cplusplus
}
#endif

#endif /* BDLM_H */
