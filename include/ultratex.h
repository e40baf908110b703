/*
 * ultratex.h -- C ABI of libultratex.so: the foreground hot path of UltraTex
 * (arXiv 2609.23169) on one AMD Instinct MI355X (gfx950).
 *
 * The path: Background Token Dropping packs the foreground tokens of the
 * unified multi-view sequence (Sec. 3.2), block lists are built from a block
 * mask (Sec. 3.3, Eq. 7), block-sparse attention runs forward and backward
 * over the packed sequence (Sec. 3.3, Eq. 8), and the packed tokens are
 * written back to the full token grid (Sec. 3.2, Eq. 4; Sec. 3.4, Eq. 9).
 *
 * Conventions shared by every call:
 *  - Pointers are DEVICE pointers unless the name ends in _host.
 *  - The caller allocates and owns every buffer; the library allocates no
 *    device memory and keeps no pointer after a call returns. Buffers must
 *    stay alive until the work queued on `stream` has completed.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL is the null
 *    stream). The only host synchronisations are the optional *_host outputs,
 *    which wait for the stream before returning.
 *  - Arguments are validated before anything is launched. On a bad argument a
 *    call returns a non-zero ut_status, launches nothing and records a message
 *    readable with ut_last_error() (per calling thread). A HIP runtime error
 *    returns UT_ERR_HIP with the HIP error text. No C++ exception crosses the
 *    ABI.
 *  - Token and block indices are int32; byte offsets are computed in 64 bits.
 *  - Block lists passed to the attention calls are trusted. With the
 *    environment variable UT_VALIDATE set (to anything but "0") those calls
 *    first copy the lists to the host, waiting for the stream, and return
 *    UT_ERR_INVALID_ARG unless every row is strictly ascending within
 *    [0, Nk) and the pointer array starts at 0 and never decreases.
 *  - bf16 is IEEE binary32 truncated to its upper 16 bits (stored as uint16),
 *    results rounded to nearest even.
 */
#ifndef ULTRATEX_H
#define ULTRATEX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define UT_ABI_VERSION 3

typedef enum {
  UT_OK = 0,
  UT_ERR_INVALID_ARG = 1, /* null / misaligned pointer, bad size or count   */
  UT_ERR_UNSUPPORTED = 2, /* a head_dim or block size the kernels lack      */
  UT_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required     */
  UT_ERR_CAPACITY = 4,    /* an output holds fewer entries than produced    */
  UT_ERR_HIP = 5          /* a HIP runtime or launch error                  */
} ut_status;

/* Element types of the foreground step calls. */
typedef enum {
  UT_BF16 = 0,
  UT_F32 = 1
} ut_dtype;

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* ut_last_error(void);

/* UT_ABI_VERSION of the loaded library. */
int ut_abi_version(void);

/* ------------------------------------------------------------------------
 * Kernel timing (a tracing aid). With tracing on, every kernel the library
 * launches is bracketed by two HIP events recorded on the stream it runs on;
 * ut_trace_read waits for those events and returns per-kernel totals in
 * first-launch order, then forgets them. Off by default. It costs two event
 * records per launch and is meant for eager launches, not graph capture.
 *
 * ut_trace_enable  on != 0 starts recording, 0 stops (records already made
 *                  stay until read). Always UT_OK.
 * ut_trace_read    consumes the records made since the last read: fills
 *                  out[0 .. min(n, max_entries)) and returns n, the number of
 *                  distinct kernels among them (entries past max_entries are
 *                  dropped; out may be NULL with max_entries = 0); -1 with
 *                  ut_last_error() set if an event could not be read (a HIP
 *                  error).
 * Names are the kernel's with its head_dim and block where it has them, e.g.
 * "bsattn_fwd<128,128>", "bwd_dkdv<128,128>", "gather_rows".
 * ---------------------------------------------------------------------- */
typedef struct {
  char name[48];
  int64_t count;      /* launches recorded */
  double total_ms;    /* summed durations */
  double min_ms;
  double max_ms;
} ut_kernel_time;
ut_status ut_trace_enable(int on);
int ut_trace_read(ut_kernel_time* out, int max_entries);

/* ------------------------------------------------------------------------
 * Background Token Dropping (Sec. 3.2, "Mask Construction and Sequence
 * Compression"): the retained set M_fg of a per-view token-grid foreground
 * mask and the Gather_{M_fg} of a full-sequence hidden state.
 *
 * fg_mask     [L] uint8, the unified sequence's token-grid masks laid out
 *             view-major then row-major; nonzero = foreground (kept).
 * x_full      [L, row_bytes] rows to gather, or NULL for the index map only.
 * row_bytes   bytes per row; a positive multiple of 16 (e.g. 3072 bf16 =
 *             6144). x_full and x_packed must be 16-byte aligned.
 * x_packed    [capacity, row_bytes] output; NULL iff x_full is NULL.
 * capacity    rows available in kept_idx and x_packed.
 * kept_idx    [capacity] int32 output: kept positions in ascending order
 *             (packed row k is full row kept_idx[k]).
 * inv_idx     [L] int32 output (NULL to skip): packed index of each position,
 *             -1 where dropped.
 * n_kept      [1] int32 device output: the number of kept positions (written
 *             even when it exceeds capacity; then only `capacity` entries are
 *             written and the host cannot tell without reading it).
 * n_kept_host optional host output: if non-NULL the call waits for the stream,
 *             stores the count, and returns UT_ERR_CAPACITY if it exceeds
 *             capacity.
 * workspace   device scratch of ut_drop_background_workspace_size(L) bytes,
 *             4-byte aligned; contents need not be initialised.
 * Errors: L < 1 or L >= 2^31, null required pointers, row_bytes not a
 *         positive multiple of 16, misalignment, capacity < 0 ->
 *         UT_ERR_INVALID_ARG; workspace too small -> UT_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
size_t ut_drop_background_workspace_size(int64_t L);
ut_status ut_drop_background(const uint8_t* fg_mask, int64_t L,
                             const void* x_full, int64_t row_bytes,
                             void* x_packed, int64_t capacity,
                             int32_t* kept_idx, int32_t* inv_idx,
                             int32_t* n_kept, int64_t* n_kept_host,
                             void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* ------------------------------------------------------------------------
 * Write-back of the packed foreground rows (Sec. 3.2, Eq. 4: only positions
 * in M_fg are updated; Sec. 3.4, Eq. 9: every other position keeps the
 * background the caller pre-filled, Gaussian noise or the tiled z_bg).
 *
 * x_packed  [n_kept, row_bytes] rows to write.
 * kept_idx  [n_kept] int32 full-sequence positions, each in [0, L); the
 *           positions must be distinct (as ut_drop_background produces).
 * row_bytes positive multiple of 16; both row buffers 16-byte aligned.
 * x_full    [L, row_bytes] in/out: row kept_idx[k] <- packed row k; rows not
 *           listed are untouched.
 * n_kept = 0 is a no-op. kept_idx contents are trusted (not range-checked).
 * ---------------------------------------------------------------------- */
ut_status ut_scatter_foreground(const void* x_packed, const int32_t* kept_idx,
                                int64_t n_kept, int64_t row_bytes, void* x_full,
                                hipStream_t stream);

/* ------------------------------------------------------------------------
 * Block index (Sec. 3.3, Eq. 7; the sets S_i of Eq. 8): from a binary block
 * mask M_c per (batch, head), the list of selected key blocks of every query
 * block (ascending j) and the transpose, the list of query blocks that select
 * each key block (ascending i), both in compressed-row form.
 *
 * block_mask [B, H, Nq, Nk] uint8, nonzero = the pair (i, j) is computed.
 * q_rowptr   [B*H*Nq + 1] int32 out: row r = (b*H + h)*Nq + i spans
 *            q_cols[q_rowptr[r] .. q_rowptr[r+1]).
 * q_cols     [cap] int32 out: key-block indices j.
 * kv_colptr  [B*H*Nk + 1] int32 out: column c = (b*H + h)*Nk + j spans
 *            kv_rows[kv_colptr[c] .. kv_colptr[c+1]).
 * kv_rows    [cap] int32 out: query-block indices i.
 * cap        entries available in q_cols and kv_rows; entries past cap are
 *            not written.
 * nnz_host   optional: if non-NULL the call waits, stores the number of
 *            nonzero mask entries, and returns UT_ERR_CAPACITY if > cap.
 * workspace  device scratch of ut_build_block_index_workspace_size(B, H, Nq,
 *            Nk) bytes. That size is 0 for every shape: the per-row and
 *            per-column counts are written straight into q_rowptr and
 *            kv_colptr and scanned there in place, so the build needs no
 *            memory beyond its outputs. NULL with workspace_bytes = 0 is
 *            valid; the arguments keep the signature uniform with the other
 *            calls that take scratch.
 * Errors: any of B, H, Nq, Nk < 1, B*H > 65535, B*H*Nq*Nk >= 2^31 (the
 *         offsets are int32), null or misaligned pointers, cap < 0 ->
 *         UT_ERR_INVALID_ARG; workspace_bytes below the required size ->
 *         UT_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
size_t ut_build_block_index_workspace_size(int32_t B, int32_t H, int32_t Nq,
                                           int32_t Nk);
ut_status ut_build_block_index(const uint8_t* block_mask, int32_t B, int32_t H,
                               int32_t Nq, int32_t Nk, int32_t* q_rowptr,
                               int32_t* q_cols, int32_t* kv_colptr,
                               int32_t* kv_rows, int64_t cap, int64_t* nnz_host,
                               void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/* ------------------------------------------------------------------------
 * Block-sparse attention forward (Sec. 3.3, Eq. 5 and Eq. 8): for each
 * (batch b, head h, query block i), O_i = softmax(Q_i K_{S_i}^T * scale)
 * V_{S_i}; key blocks outside S_i are never read.
 *
 * q, k, v   bf16 [B, N, H, D] contiguous (token-major, heads interleaved:
 *           the layout of a [N, H*D] projection output), 16-byte aligned.
 * o         bf16 [B, N, H, D] output.
 * lse       fp32 [B, H, N] output: natural-log log-sum-exp of each query
 *           row's scaled scores over its retained keys; -inf for a row whose
 *           S_i is empty (its O row is 0).
 * D         head_dim, 64 or 128. block: b_q = b_kv, 64 or 128.
 * Nq = Nk = ceil(N / block); the last block may be short (keys beyond N are
 *           excluded, rows beyond N are neither computed nor stored).
 * q_rowptr, q_cols  the row lists of ut_build_block_index for [B, H, Nq, Nq].
 *           Contents are trusted: each j must lie in [0, Nq).
 * softmax_scale  the score scale, 1/sqrt(D) in the paper; must be finite
 *           and > 0 (the kernels track the running maximum of the scaled
 *           scores, which a zero or negative scale would turn into a
 *           minimum, and mask keys with -inf scores).
 * Errors: unsupported D / block, or one sample's [N, H, D] bf16 tensor of
 *         2 GiB or more -> UT_ERR_UNSUPPORTED; N < 1, B or H < 1,
 *         null or misaligned pointers, a scale that is not finite and
 *         positive -> UT_ERR_INVALID_ARG.
 * ---------------------------------------------------------------------- */
ut_status ut_bsattn_fwd(const void* q, const void* k, const void* v, void* o,
                        float* lse, int32_t B, int32_t N, int32_t H, int32_t D,
                        int32_t block, const int32_t* q_rowptr,
                        const int32_t* q_cols, float softmax_scale,
                        hipStream_t stream);

/* ------------------------------------------------------------------------
 * Block-sparse attention backward: gradients of Eq. 8 with the block mask
 * held constant (the paper's third training stage runs this attention; it
 * prints no gradient formula). With P = softmax of the retained scores:
 * dV = P^T dO, dP = dO V^T, delta = rowsum(dO o O), dS = P o (dP - delta),
 * dQ = scale dS K, dK = scale dS^T Q. No atomics: results are deterministic.
 *
 * q, k, v, o, dout  bf16 [B, N, H, D] (o and lse from ut_bsattn_fwd).
 * lse               fp32 [B, H, N].
 * dq, dk, dv        bf16 [B, N, H, D] outputs (fully overwritten).
 * q_rowptr, q_cols, kv_colptr, kv_rows  both lists of ut_build_block_index.
 * workspace         device scratch, 16-byte aligned, of at least
 *                   ut_bsattn_bwd_workspace_size(B, N, H) bytes (8 per query
 *                   row): the row log-sum-exp in log2 units and
 *                   -delta = -rowsum(dO o O) as two planes of 4 bytes per row.
 *                   Bytes past that, from the next 256-byte boundary, hold
 *                   a flag per query block (4 bytes each), a map of 4 bytes
 *                   per pair and bf16 dS tiles of 2 block^2 bytes each (32
 *                   KiB at block 128), one per retained pair in column-list
 *                   order: the dK/dV pass writes the tiles that fit, and every
 *                   query block whose tiles all fit takes dQ from them (one
 *                   product per pair); the other query blocks recompute S and
 *                   dP (three products per pair). The row and column lists
 *                   must describe the same mask, as ut_build_block_index
 *                   makes them. ut_bsattn_bwd_workspace_size_stored(B, N, H,
 *                   block, nnz) is the size at which all nnz pairs fit.
 *                   Either way the results agree to rounding (dS is bf16 in
 *                   both).
 * Errors: as ut_bsattn_fwd, plus UT_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
size_t ut_bsattn_bwd_workspace_size(int32_t B, int32_t N, int32_t H);
/* Workspace with room for the dS tiles of nnz retained pairs (the nnz of
 * ut_build_block_index); 0 for block not 64 or 128, nnz < 0 or invalid sizes. */
size_t ut_bsattn_bwd_workspace_size_stored(int32_t B, int32_t N, int32_t H,
                                           int32_t block, int64_t nnz);
ut_status ut_bsattn_bwd(const void* q, const void* k, const void* v,
                        const void* o, const void* dout, const float* lse,
                        void* dq, void* dk, void* dv, int32_t B, int32_t N,
                        int32_t H, int32_t D, int32_t block,
                        const int32_t* q_rowptr, const int32_t* q_cols,
                        const int32_t* kv_colptr, const int32_t* kv_rows,
                        float softmax_scale, void* workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * ut_bsattn_bwd without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving or
 * training loops, harnesses that forbid hipMalloc. Arguments, outputs and
 * errors are those of ut_bsattn_bwd; the call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine) and runs the same kernels.
 *
 * Scratch: a built-in device array of 32 MiB per GPU, part of the library's
 * code object (loaded with it on each GPU the library runs on and held until
 * the process ends). It holds the 8 bytes per query row of the statistics
 * planes, so B*H*N may be at most 4,194,304 (e.g. 24 heads x 174,762
 * tokens); larger problems return UT_ERR_WORKSPACE and launch nothing. Every
 * call on one GPU shares that GPU's array: calls that overlap in time on one
 * GPU (concurrent streams, threads) race on it and must be serialised by the
 * caller. Each call writes every row it reads, so nothing needs clearing
 * between calls. The UT_VALIDATE list check is not applied here (it copies
 * the lists to the host and waits for the stream).
 * ---------------------------------------------------------------------- */
ut_status ut_bsattn_bwd_noalloc(const void* q, const void* k, const void* v,
                                const void* o, const void* dout,
                                const float* lse, void* dq, void* dk, void* dv,
                                int32_t B, int32_t N, int32_t H, int32_t D,
                                int32_t block, const int32_t* q_rowptr,
                                const int32_t* q_cols, const int32_t* kv_colptr,
                                const int32_t* kv_rows, float softmax_scale,
                                hipStream_t stream);

/* ------------------------------------------------------------------------
 * Variable-length batches of the two attention calls: B samples of differing
 * kept-token counts packed back to back in one launch. The paper buckets
 * training samples by their foreground token count (Sec. 4.1, Implementation
 * Details) because the count differs from asset to asset; packing lets one
 * launch serve a bucket whose counts still differ. Each sample attends only
 * within itself, with the same math as ut_bsattn_fwd / ut_bsattn_bwd.
 *
 * q, k, v, o, dout, dq, dk, dv  bf16 [T, H, D]: sample b holds tokens
 *           [cu_seqlens[b], cu_seqlens[b+1]).
 * cu_seqlens  device int32 [B + 1], 0 = cu[0] <= cu[1] <= ... <= cu[B] = T.
 * T         packed tokens (int64, below 2^31; T = 0 launches nothing).
 * max_seqlen  >= every sample's length; sizes the block grid:
 *           Nb = ceil(max_seqlen / block) blocks per sample.
 * lse       fp32 [H, T] (head-major over the packed tokens).
 * q_rowptr, q_cols (and kv_colptr, kv_rows)  lists of ut_build_block_index
 *           over a [B, H, Nb, Nb] block mask. Sample b uses its leading
 *           ceil(len_b / block) block rows and columns; list entries past
 *           them are ignored, and its last block may be short.
 * workspace (backward) at least ut_bsattn_bwd_varlen_workspace_size(T, H)
 *           bytes; past the next 256-byte boundary, dS tiles as in
 *           ut_bsattn_bwd (ut_bsattn_bwd_varlen_workspace_size_stored(B, T,
 *           max_seqlen, H, block, nnz) holds all of them).
 * Offsets are clamped to [0, T] and lengths to max_seqlen inside the
 * kernels, so bad offsets cannot reach outside the tensors; tokens covered by
 * no sample are left unwritten. With UT_VALIDATE set, cu_seqlens is checked
 * as described above (UT_ERR_INVALID_ARG otherwise).
 * Errors: as the uniform calls, with max_seqlen in the role of N.
 * ---------------------------------------------------------------------- */
ut_status ut_bsattn_fwd_varlen(const void* q, const void* k, const void* v,
                               void* o, float* lse, const int32_t* cu_seqlens,
                               int32_t B, int64_t T, int32_t max_seqlen,
                               int32_t H, int32_t D, int32_t block,
                               const int32_t* q_rowptr, const int32_t* q_cols,
                               float softmax_scale, hipStream_t stream);
size_t ut_bsattn_bwd_varlen_workspace_size(int64_t T, int32_t H);
size_t ut_bsattn_bwd_varlen_workspace_size_stored(int32_t B, int64_t T,
                                                  int32_t max_seqlen, int32_t H,
                                                  int32_t block, int64_t nnz);
ut_status ut_bsattn_bwd_varlen(const void* q, const void* k, const void* v,
                               const void* o, const void* dout,
                               const float* lse, void* dq, void* dk, void* dv,
                               const int32_t* cu_seqlens, int32_t B, int64_t T,
                               int32_t max_seqlen, int32_t H, int32_t D,
                               int32_t block, const int32_t* q_rowptr,
                               const int32_t* q_cols, const int32_t* kv_colptr,
                               const int32_t* kv_rows, float softmax_scale,
                               void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/* ------------------------------------------------------------------------
 * Top-K block selection (Sec. 3.3, Eq. 6 and Eq. 7): the block mask M_c of
 * block-sparse attention from mean-pooled query and key blocks. Per (b, h),
 * pool(X)_i is the mean of block i's token rows (a short last block averages
 * its real tokens), S_c = pool(Q) pool(K)^T, and row i of the mask keeps the
 * k_keep largest entries of S_c[i, :]. Equal scores are taken lower j first.
 * No block is forced (the diagonal included). The output feeds
 * ut_build_block_index.
 *
 * q, k        bf16 [B, N, H, D] contiguous, 16-byte aligned.
 * D           a multiple of 8, at most 512. block: >= 1.
 * k_keep      blocks kept per row, >= 1 (floor(rho N_k) in the paper; the
 *             caller computes it); k_keep >= Nk keeps every block.
 * prefix_blocks  P in [0, Nk]: leading blocks of always-kept tokens (the
 *             text tokens of the joint sequence, 512 in the paper's token
 *             counts): rows i < P keep every block, every row keeps blocks
 *             j < P, and the k_keep best blocks are chosen among j >= P.
 * block_mask  uint8 [B, H, Nk, Nk] output, Nk = ceil(N / block); 1 = kept.
 * workspace   device scratch of ut_topk_block_mask_workspace_size bytes
 *             (the pooled rows, fp32), 16-byte aligned.
 * Scores are fp32 (sums in order over tokens and over d); a row whose
 * k-th and (k+1)-th scores differ by less than the fp32 rounding of that
 * arithmetic may differ from an exact-arithmetic selection, and is then still
 * a valid Top-K of the fp32 scores. Inputs must be finite.
 * Errors: sizes < 1, D not a multiple of 8 or > 512, B > 65535, null or
 *         misaligned pointers, k_keep < 1, prefix_blocks outside [0, Nk] ->
 *         UT_ERR_INVALID_ARG; a row of
 *         scores too long for one workgroup's LDS (Nk + D > 16384) ->
 *         UT_ERR_UNSUPPORTED; workspace too small -> UT_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
size_t ut_topk_block_mask_workspace_size(int32_t B, int32_t N, int32_t H, int32_t D,
                                         int32_t block);
ut_status ut_topk_block_mask(const void* q, const void* k, int32_t B, int32_t N,
                             int32_t H, int32_t D, int32_t block, int32_t k_keep,
                             int32_t prefix_blocks, uint8_t* block_mask, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Foreground-only Euler update (Sec. 3.2, Eq. 4): at every retained position
 * i = kept_idx[k], z[i, :] += dt * v[k, :] with dt = t_prev - t_curr; all
 * other positions keep their values (the initial noise).
 *
 * z         fp32 [L, C] in/out, 16-byte aligned.
 * v         [n_kept, C] packed velocities, UT_BF16 or UT_F32, aligned to
 *           8 (bf16) or 16 (fp32) bytes.
 * C         channels per token, a positive multiple of 4.
 * kept_idx  [n_kept] int32, distinct positions (as ut_drop_background
 *           produces); entries outside [0, L) are skipped.
 * Each element is one fp32 fused multiply-add (one rounding). n_kept = 0 is
 * a no-op.
 * Errors: L < 1, C not a positive multiple of 4, n_kept < 0 or > L, bad
 *         dtype, non-finite dt, null or misaligned pointers ->
 *         UT_ERR_INVALID_ARG.
 * ---------------------------------------------------------------------- */
ut_status ut_euler_update_foreground(float* z, int64_t L, int64_t C, const void* v,
                                     ut_dtype v_dtype, const int32_t* kept_idx,
                                     int64_t n_kept, float dt, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Foreground flow-matching loss (Sec. 3.2, Eq. 3, with the target velocity
 * eps - z_tgt of Eq. 1-2): with i = kept_idx[k],
 *   loss = sum_{k, c} (v[k, c] - (eps[i, c] - z0[i, c]))^2 / (n_kept C)
 * (the mean over retained tokens and channels), and optionally its gradient
 *   grad[k, c] = 2 (v[k, c] - (eps[i, c] - z0[i, c])) / (n_kept C).
 *
 * v         [n_kept, C] model prediction, v_dtype.
 * eps, z0   [L, C] noise and clean target latent on the full grid, x_dtype.
 *           Rows not listed in kept_idx are never read.
 * loss      [1] fp32 device output (0 when n_kept = 0).
 * grad      [n_kept, C] fp32 device output, or NULL.
 * workspace device scratch of ut_fg_flow_loss_workspace_size() bytes,
 *           8-byte aligned (per-workgroup partial sums).
 * Differences and squares are taken in fp64 and summed in a fixed order: the
 * loss is deterministic and within a few fp64 roundings of exact before its
 * final rounding to fp32. Alignment as for ut_euler_update_foreground.
 * Errors: as ut_euler_update_foreground, plus UT_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
size_t ut_fg_flow_loss_workspace_size(void);
ut_status ut_fg_flow_loss(const void* v, ut_dtype v_dtype, const void* eps, const void* z0,
                          ut_dtype x_dtype, int64_t L, int64_t C,
                          const int32_t* kept_idx, int64_t n_kept, float* loss,
                          float* grad, void* workspace, size_t workspace_bytes,
                          hipStream_t stream);

/* ------------------------------------------------------------------------
 * Composite latent for foreground-aware decoding (Sec. 3.4, Eq. 9): row i of
 * z_mix is the denoised packed row inv_idx[i] where position i was retained,
 * and otherwise row i mod bg_rows of the canonical background latent z_bg
 * (one view's token grid, tile-repeated over the views).
 *
 * x_packed  [n_kept, row_bytes] packed rows (NULL allowed when n_kept = 0).
 * inv_idx   [L] int32, the inverse map of ut_drop_background: the packed
 *           index of each position, -1 where dropped. Entries outside
 *           [0, n_kept) take the background row.
 * z_bg      [bg_rows, row_bytes]. z_mix: [L, row_bytes] output (every row
 *           written). row_bytes: a positive multiple of 16; the row buffers
 *           16-byte aligned. A byte copy: any element type.
 * Errors: L < 1 or >= 2^31, bg_rows < 1, n_kept < 0 or > L, row_bytes not
 *         a positive multiple of 16, null or misaligned pointers ->
 *         UT_ERR_INVALID_ARG.
 * ---------------------------------------------------------------------- */
ut_status ut_composite_latent(const void* x_packed, int64_t n_kept,
                              const int32_t* inv_idx, int64_t L, const void* z_bg,
                              int64_t bg_rows, int64_t row_bytes, void* z_mix,
                              hipStream_t stream);

/* ------------------------------------------------------------------------
 * Token-grid foreground masks from alpha masks (Sec. 3.2, "Mask Construction
 * and Sequence Compression"): a token is foreground when any pixel of its
 * patch x patch block has alpha > threshold; the result is then dilated by a
 * (2 radius + 1)^2 square, clipped at each view's border. (The paper gives
 * neither rule; these are the readings taken.)
 *
 * alpha       uint8 [V, Hp, Wp], 16-byte aligned; Hp and Wp multiples of
 *             patch; patch a positive multiple of 16 (16 in the paper: the
 *             latent token grid is 1/16 of the image).
 * threshold   0..255. radius: 0..16 (0 = no dilation).
 * token_mask  uint8 [V, Hp / patch, Wp / patch] output, 1 = foreground.
 * workspace   ut_token_mask_workspace_size bytes (the undilated mask),
 *             unused (may be NULL) when radius = 0.
 * Errors: bad sizes, patch, threshold or radius, null or misaligned pointers
 *         -> UT_ERR_INVALID_ARG; workspace too small -> UT_ERR_WORKSPACE.
 * ---------------------------------------------------------------------- */
size_t ut_token_mask_workspace_size(int32_t V, int32_t Hp, int32_t Wp, int32_t patch);
ut_status ut_token_mask_from_alpha(const uint8_t* alpha, int32_t V, int32_t Hp,
                                   int32_t Wp, int32_t patch, int32_t threshold,
                                   int32_t radius, uint8_t* token_mask, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* ULTRATEX_H */
