/*
 * shc.h -- sparse contact-layer operators on one AMD Instinct MI355X (gfx950).
 *
 * C ABI of libshc.so.  The operators follow Sec. 3 of "Efficient Human-Contact
 * Representation for Human-Scene Interaction" (ECO, arXiv 2608.09388):
 *
 *   Eq. 1    a 0/1 contact mask multiplies the per-vertex input;
 *   Eq. 2    the masked tensor is decomposed into a coordinate list C' of
 *            (frame/body b, vertex v) pairs and the compact feature rows S';
 *   Eqs. 4-5 the sparse convolution is evaluated only at active centre
 *            coordinates, summing slot weight x neighbour feature over the
 *            kernel slots whose neighbour is present in C;
 *   Eq. 6    the sparse linear layer maps every feature row, C unchanged;
 *   Eq. 10   activations act elementwise on the rows, C unchanged;
 *   pooling  (named with the sparse layers, Sec. 3.2) is a per-body maximum.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All array arguments are DEVICE pointers (memory on the current HIP device)
 *   unless the comment says "host".  The caller owns every buffer; the library
 *   keeps no pointer after the work it enqueues has run, allocates nothing and
 *   holds no state between calls (the exceptions: the stream-ordering events
 *   of shc_event_create and the stack executors of shc_stack_create, which
 *   the caller creates and destroys).
 * - Every call validates its arguments on the host, then enqueues its kernels
 *   on `stream` and returns without waiting (the one exception is the optional
 *   host count of shc_compact_mask).  Calls are thread-safe.
 * - Layouts are row-major and contiguous.  Feature rows hold C channels of
 *   `dtype`: SHC_F32 (IEEE binary32) or SHC_BF16 (bfloat16 stored as uint16).
 *   Features, weights and outputs of one call share the dtype; bias is always
 *   fp32; products are accumulated in fp32; bf16 outputs are rounded to
 *   nearest, ties to even.
 * - Every device pointer must be 16-byte aligned (SHC_ERR_MISALIGNED), and
 *   channel counts must be multiples of 16 in [16, 4096] (SHC_ERR_UNSUPPORTED).
 * - Index arrays are int32.  C' is ordered by (b, v) ascending; inv[b*V + v]
 *   is the row of (b, v) in C' or -1; row_ptr[b] is the first row of body b
 *   and row_ptr[B] = N'.  B*V must be below 2^31.
 * - Index entries outside their valid range (a neighbour outside [-1, V), an
 *   inv entry outside [-1, n_rows), a coordinate outside [0, B) x [0, V)) are
 *   treated as absent rows, never dereferenced.
 * - Inputs and outputs of one call must not overlap.
 * - Return value: SHC_OK (0) or a negative SHC_ERR_* code.  Nothing is
 *   launched when validation fails.  SHC_ERR_HIP reports a HIP runtime or
 *   launch failure; shc_last_error() then holds the message (thread-local).
 */
#ifndef SHC_H_
#define SHC_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* dtype codes */
#define SHC_F32 0
#define SHC_BF16 1

/* activation codes (Eq. 10) */
#define SHC_ACT_NONE 0
#define SHC_ACT_RELU 1 /* y if y > 0 else 0 */

/* status codes */
#define SHC_OK 0
#define SHC_ERR_INVALID_ARG (-1) /* NULL pointer, negative or zero size, bad flag */
#define SHC_ERR_CAPACITY (-2)    /* workspace too small, or N' above `cap` */
#define SHC_ERR_MISALIGNED (-3)  /* a device pointer is not 16-byte aligned */
#define SHC_ERR_UNSUPPORTED (-4) /* channels not a multiple of 16, K > 32, dtype/act code */
#define SHC_ERR_HIP (-5)         /* HIP runtime or launch failure */

/* Human-readable name of a status code (static string, never NULL). */
const char* shc_status_string(int status);

/* Detail of the last failure on this thread ("" if none). */
const char* shc_last_error(void);

/* Bytes of device workspace shc_compact_mask needs for a B x V mask. */
size_t shc_compact_mask_workspace(int32_t B, int32_t V);

/*
 * Mask compaction -- the decomposition of Eq. 2 (Sec. 3.1), for the per-vertex
 * mask of Eq. 1 given per body/frame.
 *
 *   mask      [B*V] uint8, entry (b, v) is active when non-zero.
 *   coords    [cap][2] int32 out: row i of C' is (b_i, v_i), rows in (b, v)
 *             ascending order; only the first min(N', cap) rows are written.
 *   inv       [B*V] int32 out: row of (b, v) in C', or -1.  Entries whose row
 *             would be >= cap are still written with that row number.
 *   row_ptr   [B+1] int32 out: first row of every body, row_ptr[B] = N'.
 *   n_active_dev  [1] int32 out: N'.
 *   n_active_host host int64*, may be NULL.  When set, the call waits for the
 *             stream, stores N' there and returns SHC_ERR_CAPACITY if N' > cap.
 *             If it lies in page-locked host memory mapped into the device
 *             (hipHostMalloc), the kernel stores the count there itself and
 *             the call returns as soon as the count has arrived: the other
 *             outputs may still be being written, and work enqueued later on
 *             the same stream is ordered after them (synchronise the stream
 *             before reading them on the host).  Pageable memory costs one
 *             device-to-host copy and a full stream synchronisation.
 *   cap       rows available in `coords` (>= 0).
 *   ws, ws_bytes  device workspace of at least shc_compact_mask_workspace(B, V)
 *             bytes; its contents on entry do not matter.
 * Results are deterministic and bit-exact (integer work only).
 */
int shc_compact_mask(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords, int32_t* inv,
                     int32_t* row_ptr, int32_t* n_active_dev, int64_t* n_active_host, int64_t cap,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * shc_compact_mask without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The compaction's per-span counts go to a
 * scratch array of 64 KB that the library holds in device memory, one copy
 * per GPU, kept until the process ends; a B x V mask needs
 * shc_compact_mask_workspace(B, V) bytes of it (at most 4 KB for any mask the
 * library takes), and a mask that needed more would get SHC_ERR_CAPACITY.
 * The call makes no allocation of its own (no hipMalloc, hipFree or
 * allocating library routine); for none at all, pass n_active_host as NULL
 * or in page-locked memory (pageable memory goes through a HIP copy).
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (concurrent streams, or host threads) race and must be ordered by the
 * caller.  Nothing in the array needs to start at any value.  Arguments,
 * outputs, waiting and errors otherwise as for shc_compact_mask.
 */
int shc_compact_mask_noalloc(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                             int32_t* inv, int32_t* row_ptr, int32_t* n_active_dev,
                             int64_t* n_active_host, int64_t cap, hipStream_t stream);

/*
 * shc_compact_mask in two halves, for a caller with work to enqueue before it
 * needs N' (work that reads only inv, such as shc_clear_inactive_rows):
 *
 * shc_compact_mask_start -- the same compaction, launched on `stream` without
 *   waiting.  n_active_host must lie in page-locked host memory mapped into
 *   the device (hipHostMalloc), else SHC_ERR_INVALID_ARG: the call stores -1
 *   there and the kernel stores N' as soon as it is known.  Other arguments
 *   and outputs as for shc_compact_mask.
 * shc_compact_mask_wait -- waits until that count has arrived in
 *   *n_active_host (leaving it there); SHC_ERR_CAPACITY if N' > cap (the cap
 *   given to the start call), SHC_ERR_HIP if the stream fails or drains
 *   without a count.  The other outputs may still be being written; work
 *   enqueued on the stream is ordered after them.
 */
int shc_compact_mask_start(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                           int32_t* inv, int32_t* row_ptr, int32_t* n_active_dev,
                           int64_t* n_active_host, int64_t cap, void* ws, size_t ws_bytes,
                           hipStream_t stream);
int shc_compact_mask_wait(int64_t* n_active_host, int64_t cap, hipStream_t stream);

/*
 * shc_compact_mask_table_start -- shc_compact_mask_start that also writes the
 *   neighbour-row table of the active set (shc_build_neighbor_table's output
 *   for the N' rows it produces) in the same pass, so the table needs no
 *   launch of its own and no host knowledge of N':
 *     nbr    [V][K] int32 neighbour lists, -1 = none (as for the table call);
 *     table  [K][N'] int32 out, slot-major with row stride N'; written only
 *            when N' <= cap, so it must hold K * cap entries (may be NULL when
 *            cap = 0).
 *   K in [1, 32]; V <= 19456 (a body's row numbering is kept on chip),
 *   else SHC_ERR_UNSUPPORTED.  Finish with shc_compact_mask_wait.  Other
 *   arguments, outputs and errors as for shc_compact_mask_start.
 */
int shc_compact_mask_table_start(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                                 int32_t* inv, int32_t* row_ptr, int32_t* n_active_dev,
                                 int64_t* n_active_host, int64_t cap, const int32_t* nbr,
                                 int32_t K, int32_t* table, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * Gather of the active feature rows -- S' of Eq. 2: S[i] = x[b_i * V + v_i].
 *
 *   x       [B*V][C] dense per-vertex features.
 *   coords  [n_rows][2] from shc_compact_mask.
 *   S       [n_rows][C] out.
 * An exact copy; rows whose coordinate is out of range are written as zeros.
 */
int shc_gather_rows(const void* x, const int32_t* coords, int64_t n_rows, int32_t B, int32_t V,
                    int32_t C, int32_t dtype, void* S, hipStream_t stream);

/*
 * Several masks applied to the same input (Sec. 3.1), stacked as a batch
 * axis: mask k of body b is body b' = k * B + b of a [kappa * B][V] mask
 * (compacted by shc_compact_mask like any other), and every layer call then
 * takes kappa * B bodies unchanged.
 *
 * shc_gather_rows_stacked -- S[i] = x[(b'_i mod B) * V + v_i]: the rows of
 *   the stacked batch read the input of their own body.  x [B*V][C]; coords
 *   [n_rows][2] with b' in [0, kappa * B) (others read zeros).  An exact copy.
 * shc_combine_stacked -- combines kappa stacked outputs, row by row and
 *   channel by channel (the paper leaves the rule open):
 *     out[r] = op over k < kappa of Y[k * rows + r],   r < rows,
 *   op = SHC_COMBINE_SUM, SHC_COMBINE_MEAN (the sum divided by kappa) or
 *   SHC_COMBINE_MAX.  Y [kappa * rows][C] (e.g. dense outputs with rows =
 *   B*V, or pooled outputs with rows = B), out [rows][C].  Sums are taken in
 *   fp32 in k order and rounded once; the maximum is exact (inputs are
 *   numbers).
 */
int shc_gather_rows_stacked(const void* x, const int32_t* coords, int64_t n_rows, int32_t B,
                            int32_t kappa, int32_t V, int32_t C, int32_t dtype, void* S,
                            hipStream_t stream);
#define SHC_COMBINE_SUM 0
#define SHC_COMBINE_MEAN 1
#define SHC_COMBINE_MAX 2
int shc_combine_stacked(const void* Y, int32_t kappa, int64_t rows, int32_t C, int32_t dtype,
                        int32_t op, void* out, hipStream_t stream);

/*
 * A mask drawn per element (vertex and channel) instead of per vertex:
 *
 * shc_row_mask_from_elements -- m[b*V + v] = 1 when any of the C bytes
 *   me[(b*V + v)*C + c] is non-zero, else 0: the vertex activity that
 *   shc_compact_mask then takes.  me [B*V][C] uint8, m [B*V] uint8.
 * shc_gather_rows_masked -- S[i][c] = x[(b_i V + v_i)][c] where
 *   me[(b_i V + v_i)][c] is non-zero, else 0: the gathered rows multiplied by
 *   the element mask.  Arguments as for shc_gather_rows plus me.
 */
int shc_row_mask_from_elements(const uint8_t* me, int32_t B, int32_t V, int32_t C, uint8_t* m,
                               hipStream_t stream);
int shc_gather_rows_masked(const void* x, const uint8_t* me, const int32_t* coords,
                           int64_t n_rows, int32_t B, int32_t V, int32_t C, int32_t dtype,
                           void* S, hipStream_t stream);

/*
 * Sparse linear layer -- Eq. 6 (+ Eq. 10): out[i] = act(S[i] W + bias).
 *
 *   S     [n_rows][Cin] active feature rows (coordinates unchanged, C' = C).
 *   W     [Cin][Cout] (row-major: W[k][n] multiplies channel k into output n).
 *   bias  [Cout] fp32, or NULL for none.
 *   out   [n_rows][Cout].
 * n_rows = 0 is a no-op.
 */
int shc_sparse_linear(const void* S, int64_t n_rows, const void* W, const float* bias, int32_t Cin,
                      int32_t Cout, int32_t dtype, int32_t act, void* out, hipStream_t stream);

/*
 * Gather fused into the sparse linear layer -- Eq. 2 then Eq. 6 (+ Eq. 10):
 *
 *   out[i] = act(x[b_i * V + v_i] W + bias)
 *
 * the result of shc_gather_rows followed by shc_sparse_linear (bit for bit
 * when both calls take the same kernel), without writing the gathered rows.
 *   x       [B*V][Cin] dense per-vertex features; coords [n_rows][2] from
 *           shc_compact_mask (a coordinate outside [0,B)x[0,V) reads zeros).
 *   W, bias, out, act as for shc_sparse_linear; out must not overlap x.
 * n_rows = 0 is a no-op.
 */
int shc_gather_sparse_linear(const void* x, const int32_t* coords, int64_t n_rows, int32_t B,
                             int32_t V, const void* W, const float* bias, int32_t Cin,
                             int32_t Cout, int32_t dtype, int32_t act, void* out,
                             hipStream_t stream);

/*
 * Sparse neighbourhood (spiral / k-NN) convolution -- Eqs. 4-5 (+ Eq. 10),
 * output only at the active rows:
 *
 *   out[i] = act( bias + sum_{j<K} S[r_ij] W[j] ),
 *   r_ij   = inv[b_i * V + nbr[v_i * K + j]]; a slot adds nothing when its
 *            neighbour is -1 or the neighbour vertex is inactive (r_ij = -1).
 *
 *   S       [n_rows][Cin] active rows, coords/inv from shc_compact_mask.
 *   nbr     [V][K] int32 neighbour vertex of every slot, -1 for none.  The
 *           mesh is shared by all bodies.  Slot j plays the part of kernel
 *           position j of Eq. 4; the centre vertex is simply the slot whose
 *           entry is v itself.
 *   W       [K][Cin][Cout]: a Cin x Cout channel-mixing matrix per slot (the
 *           paper's scalar slot weight w_j is the case W[j] = w_j * I).
 *   bias    [Cout] fp32 or NULL.   K in [1, 32].
 *   out     [n_rows][Cout], must not overlap S.
 * n_rows = 0 is a no-op.
 */
int shc_sparse_neighbor_conv(const void* S, const int32_t* coords, const int32_t* inv,
                             int64_t n_rows, int32_t B, int32_t V, const int32_t* nbr, int32_t K,
                             const void* W, const float* bias, int32_t Cin, int32_t Cout,
                             int32_t dtype, int32_t act, void* out, hipStream_t stream);

/*
 * Neighbour-row table of an active set -- the index sets of Eqs. 4-5 in
 * compact row numbers, built once per mask:
 *
 *   table[j * n_rows + i] = r_ij = inv[b_i * V + nbr[v_i * K + j]], or -1
 *
 * for every active row i < n_rows and slot j < K (slot-major: row stride
 * n_rows).  The active set is the same for every layer (C' = C), so every
 * convolution over this mask can read the table instead of rebuilding it.
 *
 *   coords, inv  from shc_compact_mask (n_rows = N').
 *   nbr     [V][K] as for shc_sparse_neighbor_conv; entries outside [0, V)
 *           and inactive neighbours give -1.
 *   table   [K][n_rows] int32 out, device memory owned by the caller.
 * n_rows = 0 is a no-op.  Results are exact and deterministic.
 */
int shc_build_neighbor_table(const int32_t* coords, const int32_t* inv, int64_t n_rows,
                             int32_t B, int32_t V, const int32_t* nbr, int32_t K, int32_t* table,
                             hipStream_t stream);

/*
 * Sparse neighbourhood convolution reading its index sets from a table built
 * by shc_build_neighbor_table for the same active set (same n_rows, K):
 *
 *   out[i] = act( bias + sum_{j<K} S[table[j * n_rows + i]] W[j] ),
 *
 * a slot whose entry is outside [0, n_rows) adding nothing.  Same result as
 * shc_sparse_neighbor_conv on the mask the table came from; arguments as
 * there, with `table` in place of coords / inv / nbr / B / V.
 */
int shc_sparse_neighbor_conv_table(const void* S, const int32_t* table, int64_t n_rows,
                                   int32_t K, const void* W, const float* bias, int32_t Cin,
                                   int32_t Cout, int32_t dtype, int32_t act, void* out,
                                   hipStream_t stream);

/*
 * Conv plan of an active set.  The weight-stationary conv splits the active
 * rows into row groups (one workgroup each, per column slice of W) and, in
 * every workgroup, first builds the group's index lists from the table: the
 * rows sorted by their first sparse slot, each wavefront's list of
 * (16-row block, slot) jobs.  These depend only on the table and the shape,
 * so one plan, built once, serves every column slice and every conv layer of
 * the same shape on that active set (the layers of Eqs. 4-5 stacked on one
 * mask).  A planned layer computes the same per-row sums in the same order as
 * shc_sparse_neighbor_conv_table, so its output is identical to that call's.
 *
 * shc_conv_plan_max_rows: the largest active-row count whose conv with K
 *   slots and Cin -> Cout channels of dtype takes a plan on the current
 *   device (every smaller count does too); 0 when none does (fp32, a shape
 *   the weight-stationary kernel does not run, invalid arguments, no
 *   device).  Past it the conv runs on the tiled kernel, which builds no
 *   index lists: use shc_sparse_neighbor_conv_table there.
 *
 * shc_conv_plan_bytes: bytes of a plan buffer that holds the plan of any
 *   active set of at most n_rows rows (those up to shc_conv_plan_max_rows),
 *   for that shape on the current device; 0 when none takes a plan.  A
 *   multiple of 1024.
 *
 * shc_build_conv_plan: writes the plan of `table` (from
 *   shc_build_neighbor_table or shc_compact_mask_table_start, [K][n_rows])
 *   for layers of shape (n_rows, K, Cin, Cout, dtype) into `plan`, a device
 *   buffer of plan_bytes >= shc_conv_plan_bytes(n_rows, ...) bytes
 *   (caller-owned, 16-byte aligned; the plan of n_rows rows may take fewer:
 *   the bytes past it are not touched).  Stream-ordered; reads only `table`.
 *
 * shc_sparse_neighbor_conv_planned: the conv of shc_sparse_neighbor_conv_table
 *   with the index lists taken from `plan` (built by shc_build_conv_plan for
 *   the same active set and the same n_rows, K, Cin, Cout, dtype; the table
 *   itself is not read).  Other arguments as there.
 *
 * Errors: the calls' shape errors are those of shc_sparse_neighbor_conv_table;
 * SHC_ERR_UNSUPPORTED when the shape (n_rows included) takes no plan,
 * SHC_ERR_CAPACITY when plan_bytes is below that plan's size.  A plan of another active set or shape is not
 * detected: the result is then wrong, but every access stays inside S, W,
 * bias, out and the plan.
 */
/*
 * The conv of shc_sparse_neighbor_conv_table with slot 0 and the other slots
 * computed apart (Eqs. 4-5 with Eq. 10's activation; the slots of a row are
 * summed in a different order, so results agree to rounding, not bit for
 * bit):
 *
 *   P[j][i] = S[table[j][i]] W[j]   for every present (i, j >= 1), in fp32,
 *   out[i]  = act( P[j1][i] + bias + P[j2][i] + ... + S[table[0][i]] W[0] ),
 *
 * j1 < j2 < ... the row's present slots j >= 1, slot 0's product accumulated
 * last.  Two launches: one multiplies the present (row, slot) pairs of every
 * slot j >= 1 by W[j], 16 pairs per matrix-core job, into the workspace; the
 * other computes slot 0 for every row and adds the row's partial rows.  Each
 * weight matrix and each neighbour row then reaches a compute unit once for
 * all output columns, which pays when few pairs are present (sparse masks)
 * and rows are wide: for 256 channels the table conv re-reads the weights for
 * every 128-row tile.  Slot 0 should be the vertex itself (spiral and k-NN
 * neighbourhoods); any other table is still computed correctly.
 *
 * shc_conv_split_workspace_bytes: bytes of the workspace of a call with up
 *   to n_rows rows: (K - 1) * n_rows * Cout * 4 (at least 16); 0 when the
 *   shape takes no split conv (dtype other than bf16, Cin or Cout outside
 *   {64, 128, 256}, K outside [1, 32], or a workspace of 2^31 bytes or more).
 * shc_sparse_neighbor_conv_split: S, table, W, bias, out, act as for
 *   shc_sparse_neighbor_conv_table; workspace: device memory of at least
 *   shc_conv_split_workspace_bytes(n_rows, ...) bytes, 16-byte aligned,
 *   owned by the caller; its contents on entry do not matter and on return
 *   are unspecified.  Stream-ordered; calls that share a workspace must not
 *   overlap.
 *
 * Errors: those of shc_sparse_neighbor_conv_table; SHC_ERR_UNSUPPORTED for a
 * shape without a split conv, SHC_ERR_CAPACITY when workspace_bytes is too
 * small.
 */
size_t shc_conv_split_workspace_bytes(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout,
                                      int32_t dtype);
int shc_sparse_neighbor_conv_split(const void* S, const int32_t* table, int64_t n_rows,
                                   int32_t K, const void* W, const float* bias, int32_t Cin,
                                   int32_t Cout, int32_t dtype, int32_t act, void* out,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Sparse neighbourhood conv with pre-arranged weights (Eqs. 4-5, with the
 * activation of Eq. 10), bf16: the same y_i as shc_sparse_neighbor_conv_table,
 *
 *   out[i] = act( bias + sum_{j < K, table[j][i] present} S[table[j][i]] W[j] ),
 *
 * summed in fp32 per row with slot 0 first and the other present slots
 * ascending.  Every slot's weights stay in the matrix cores' operand
 * registers for the whole launch, one workgroup per compute unit over a chunk
 * of consecutive active rows: the chunk's input rows are read once into LDS,
 * rows are grouped by the slots they have, and only neighbour rows outside
 * the chunk are gathered again.  Shapes: bf16, Cin and Cout in {64, 128},
 * 1 <= K <= 9.
 *
 * shc_conv_packed_weights_bytes: bytes of the packed weights of a shape,
 *   K * Cin * Cout * 2; 0 when the shape has no packed conv.
 * shc_pack_conv_weights: W [K][Cin][Cout] bf16 (device) -> Wp (device, at
 *   least shc_conv_packed_weights_bytes bytes, 16-byte aligned, owned by the
 *   caller).  For slot j, 16-column block ct and 32-channel step ks, Wp holds
 *   the 64 lanes' 16-byte operand fragments of a 16x16x32 matrix-core step
 *   contiguously: lane 16 g + i gets W[j][32 ks + 8 g + e][16 ct + i], e < 8.
 *   Pack once per weight update; stream-ordered, no host wait.
 * shc_sparse_neighbor_conv_packed: S, table, bias, out, act as for
 *   shc_sparse_neighbor_conv_table; Wp from shc_pack_conv_weights of the same
 *   K, Cin, Cout.  Table entries outside [0, n_rows) count as absent.
 *   Stream-ordered, no host wait, allocates nothing.
 *
 * Errors: those of shc_sparse_neighbor_conv_table; SHC_ERR_UNSUPPORTED for a
 * shape without a packed conv or a table of 2^31 bytes or more,
 * SHC_ERR_CAPACITY when Wp_bytes is too small.
 */
size_t shc_conv_packed_weights_bytes(int32_t K, int32_t Cin, int32_t Cout, int32_t dtype);
int shc_pack_conv_weights(const void* W, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype,
                          void* Wp, size_t Wp_bytes, hipStream_t stream);
int shc_sparse_neighbor_conv_packed(const void* S, const int32_t* table, int64_t n_rows,
                                    int32_t K, const void* Wp, const float* bias, int32_t Cin,
                                    int32_t Cout, int32_t dtype, int32_t act, void* out,
                                    hipStream_t stream);

/*
 * The packed conv's plan (Sec. 3.2: the index sets C'_k = C_k are the same
 * for every layer, so the grouping of the active rows by their slots is a
 * property of the active set, not of a layer): shc_build_conv_packed_plan
 * does the packed conv's grouping of each chunk of rows (the rows' order,
 * every (row, slot) entry as the LDS row to read, the neighbour rows to
 * stage, the staging rounds) and writes it to `plan`;
 * shc_sparse_neighbor_conv_packed_planned then computes the layer from it,
 * without the table, with the same result as shc_sparse_neighbor_conv_packed
 * on that table.  Build once per active set (after the table), on any
 * stream ordered before the layers that read it.
 *
 * shc_conv_packed_plan_bytes: bytes of a plan buffer that holds the plan of
 *   any row count up to n_rows on the current device (0: no packed conv for
 *   the shape).
 * shc_build_conv_packed_plan: table [K][n_rows] as for
 *   shc_sparse_neighbor_conv_table; plan: device memory of at least the bytes
 *   the call's n_rows needs (shc_conv_packed_plan_bytes(n_rows, ...) is
 *   enough), 16-byte aligned, owned by the caller.  Stream-ordered.
 * shc_sparse_neighbor_conv_packed_planned: S, bias, out, act as for
 *   shc_sparse_neighbor_conv_packed; plan from shc_build_conv_packed_plan of
 *   the same n_rows, K, Cin and Cout.  A chunk whose plan was built for
 *   another row count is skipped (its rows are not written); a plan of another
 *   table of the same row count gives wrong values but no access out of
 *   range.  Stream-ordered, allocates nothing.
 *
 * Errors: those of shc_sparse_neighbor_conv_packed; SHC_ERR_CAPACITY when
 * plan_bytes is below what the call's n_rows needs.
 */
size_t shc_conv_packed_plan_bytes(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout,
                                  int32_t dtype);
int shc_build_conv_packed_plan(const int32_t* table, int64_t n_rows, int32_t K, int32_t Cin,
                               int32_t Cout, int32_t dtype, void* plan, size_t plan_bytes,
                               hipStream_t stream);
int shc_sparse_neighbor_conv_packed_planned(const void* S, const void* plan, size_t plan_bytes,
                                            int64_t n_rows, int32_t K, const void* Wp,
                                            const float* bias, int32_t Cin, int32_t Cout,
                                            int32_t dtype, int32_t act, void* out,
                                            hipStream_t stream);

int64_t shc_conv_plan_max_rows(int32_t K, int32_t Cin, int32_t Cout, int32_t dtype);
size_t shc_conv_plan_bytes(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype);
int shc_build_conv_plan(const int32_t* table, int64_t n_rows, int32_t K, int32_t Cin,
                        int32_t Cout, int32_t dtype, void* plan, size_t plan_bytes,
                        hipStream_t stream);
int shc_sparse_neighbor_conv_planned(const void* S, const void* plan, size_t plan_bytes,
                                     int64_t n_rows, int32_t K, const void* W,
                                     const float* bias, int32_t Cin, int32_t Cout,
                                     int32_t dtype, int32_t act, void* out,
                                     hipStream_t stream);

/*
 * Scatter back to the dense per-vertex layout (C' = C, so row i returns to
 * (b_i, v_i)):
 *
 *   zero_fill = 1: D[r] = S[inv[r]] if inv[r] >= 0 else 0, for all r < B*V
 *                  (D = y (.) m, every row of D written).
 *   zero_fill = 0: D[b_i * V + v_i] = S[i] for i < n_rows; the rows of inactive
 *                  vertices are left untouched.
 *   S [n_rows][C], D [B*V][C].  An exact copy.
 */
int shc_scatter(const void* S, const int32_t* inv, const int32_t* coords, int64_t n_rows,
                int32_t B, int32_t V, int32_t C, int32_t dtype, int32_t zero_fill, void* D,
                hipStream_t stream);

/*
 * The zero-filled scatter (D = y (.) m, Sec. 3.2) as an update of a dense
 * output that holds the previous batch's: when D holds the zero_fill = 1
 * result of shc_scatter for a previous active set whose coordinates are
 * prev_coords [prev_rows][2], this call leaves D holding the zero_fill = 1
 * result for this set (S, inv, coords, n_rows):
 *
 *   D[b * V + v] = 0   for every (b, v) of prev_coords with inv[b * V + v] < 0,
 *   D[b_i * V + v_i] = S[i]   for every i < n_rows,
 *
 * every other row untouched.  It touches only the rows of the two active
 * sets (about 2 N' rows instead of B * V).  A dense output kept resident from
 * batch to batch starts as all zeros with prev_rows = 0.  prev_coords must
 * not be this call's coords buffer (SHC_ERR_INVALID_ARG); the caller keeps a
 * copy of the coordinates for the next call.  Coordinates out of range are
 * skipped.  Other arguments as for shc_scatter; an exact copy.
 */
int shc_scatter_update(const void* S, const int32_t* inv, const int32_t* coords, int64_t n_rows,
                       const int32_t* prev_coords, int64_t prev_rows, int32_t B, int32_t V,
                       int32_t C, int32_t dtype, void* D, hipStream_t stream);

/*
 * The zeros of the zero-filled scatter (D = y (.) m, Sec. 3.2), which need
 * only the inverse map:
 *
 *   D[r] = 0 for every r < B*V with inv[r] < 0; the other rows untouched.
 *
 * Followed by shc_scatter with zero_fill = 0 this gives shc_scatter's
 * zero_fill = 1 result for a consistent compaction (inv and coords from the
 * same shc_compact_mask, N' <= cap), and it can run before N' is known.
 *   inv [B*V] int32, D [B*V][C] of `dtype`.
 */
int shc_clear_inactive_rows(const int32_t* inv, int32_t B, int32_t V, int32_t C, int32_t dtype,
                            void* D, hipStream_t stream);

/*
 * Sparse group normalization per body/frame -- Eqs. 7-9 (Sec. 3.2): for every
 * body b and group g of C/G consecutive channels,
 *
 *   mu  = mean of the group's values over rows row_ptr[b] <= i < row_ptr[b+1]
 *   var = mean of (value - mu)^2 over the same values (biased, 1/N)
 *   out = (value - mu) / sqrt(var + eps)
 *
 * Only the active rows enter the statistics (a body's rows are its active
 * vertices), so this is not the dense normalization of the masked tensor.
 * No affine term.  G = 1 is layer normalization.
 *
 *   S [n_rows][C], row_ptr [B+1] (bounds clamped to [0, n_rows]), out
 *   [n_rows][C] of the same dtype, must not overlap S.  G must divide C; eps
 *   must be positive and finite (1e-5 is the usual value).
 * Two passes: the mean, accumulated in fp64, then the squared deviations
 * from it, summed in fp32 over at most 16 rows per thread and in fp64 beyond.
 * Each output is computed in fp32 from the mean as two fp32 terms (about
 * 12 * 2^-24 relative error in all); bf16 outputs are then rounded to
 * nearest even.
 */
int shc_segment_group_norm(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                           int32_t C, int32_t G, float eps, int32_t dtype, void* out,
                           hipStream_t stream);

/*
 * Mask scores -- Eq. 3 (Sec. 3.1) -- and the top-kappa masks kept at
 * inference.  For K masks with aligned outputs O_k [N][C] (the same N rows,
 * e.g. the dense per-vertex outputs of every body), stored mask-major as
 * O [K][N][C] bf16:
 *
 *   F[i][k]      = || O_i^T O_k ||_F^2
 *   sim[i][k]    = F[i][k] / sqrt(F[i][i] * F[k][k]), or 1 where that
 *                  denominator is 0 (a mask whose output is all zero earns
 *                  no dissimilarity credit, so it ranks last among equals)
 *   alpha_out[k] = alpha_in[k] + 1/(K-1) * sum_{i != k} (1 - sim[i][k])
 *                  (alpha_in[k] itself when K = 1)
 *   top[r]       = the mask of rank r by alpha_out, largest first, ties to
 *                  the lower index, for r < kappa.
 *
 *   alpha_in [K] fp64 or NULL (zeros); alpha_out [K] fp64; sim [K][K] fp64
 *   or NULL; top [kappa] int32 (may be NULL when kappa = 0); all device
 *   memory.  K in [1, 64]; C a multiple of 64 in [64, 1024]; bf16 only.
 *   ws, ws_bytes: device workspace of at least shc_mask_scores_workspace
 *   bytes (0 for unsupported shapes); contents on entry do not matter.
 * The Gram blocks are accumulated in fp32 by MFMA over row splits whose sums
 * are combined in a fixed order in fp64: results repeat bit for bit.
 */
size_t shc_mask_scores_workspace(int32_t K, int64_t N, int32_t C);
int shc_mask_scores(const void* O, int32_t K, int64_t N, int32_t C, int32_t dtype,
                    const double* alpha_in, double* alpha_out, double* sim, int32_t kappa,
                    int32_t* top, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Segmented max-pool per body/frame -- the sparse pooling layer (Sec. 3.2):
 *
 *   P[b][c] = max over row_ptr[b] <= i < row_ptr[b+1] of S[i][c]
 *   (IEEE maxNum: a NaN loses to any number), or `empty_value` for a body
 *   without active rows.  Segment bounds are clamped to [0, n_rows).
 *
 *   S [n_rows][C], row_ptr [B+1], P [B][C] out (same dtype as S; empty_value
 *   is converted to it).  Exact (a selection, no rounding).
 */
int shc_segment_maxpool(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                        int32_t C, int32_t dtype, float empty_value, void* P, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Backward of the sparse linear layer (Eq. 6) and the sparse neighbourhood   */
/* convolution (Eqs. 4-5), with the ReLU of Eq. 10.                           */
/* ------------------------------------------------------------------------ */

/* Virtual slots of a transposed neighbour list (see shc_transpose_neighbors). */
#define SHC_MAX_VIRTUAL_SLOTS 64

/*
 * Transposed neighbour lists of a mesh, built once per mesh.  For vertex u
 * and slot j, the vertices v with nbr[v][j] = u, ascending, are u's senders
 * through slot j; the c-th of them sits in virtual slot s = off_j + c, where
 * off_j = sum_{j' < j} m_j' and m_j is the largest number of senders any
 * vertex has through slot j.  Kt = sum_j m_j.
 *
 *   nbr [V][K] int32 (entries outside [0, V) mean "no neighbour");
 *   nbr_t [V][SHC_MAX_VIRTUAL_SLOTS] int32 out: the first V * Kt entries hold
 *     [V][Kt] (sender vertex or -1), the rest -1;
 *   slot_of [SHC_MAX_VIRTUAL_SLOTS] int32 out: the slot j of virtual slot s
 *     (-1 past Kt);
 *   *Kt_host out (host memory): Kt.  The call waits for the stream.
 *   ws: device workspace of shc_transpose_neighbors_workspace(V, K) bytes.
 * K <= 32; a mesh with Kt > SHC_MAX_VIRTUAL_SLOTS gets SHC_ERR_UNSUPPORTED.
 */
size_t shc_transpose_neighbors_workspace(int32_t V, int32_t K);
int shc_transpose_neighbors(const int32_t* nbr, int32_t V, int32_t K, int32_t* nbr_t,
                            int32_t* slot_of, int32_t* Kt_host, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/*
 * Transposed table of an active set (the companion of
 * shc_build_neighbor_table): for active row r = (b, u) and virtual slot s,
 *
 *   table_t[s * n_rows + r] = inv[b * V + nbr_t[u * Kt + s]], or -1,
 *
 * the active row that sends to r through s; row_slots[r] has bit s set when
 * that entry is a row.  coords, inv: from shc_compact_mask; table_t
 * [Kt][n_rows] int32 and row_slots [n_rows] uint64 out.  Kt <= 64.
 */
int shc_build_transposed_table(const int32_t* coords, const int32_t* inv, int64_t n_rows,
                               int32_t B, int32_t V, const int32_t* nbr_t, int32_t Kt,
                               int32_t* table_t, uint64_t* row_slots, hipStream_t stream);

/*
 * Gradients of the sparse linear layer out = act(S W + b) (Eq. 6, Eq. 10):
 *
 *   dZ = dY (.) [Y > 0] with act = SHC_ACT_RELU (dZ = dY without),
 *   dS = dZ W^T,   dW = S^T dZ,   db = sum over rows of dZ,
 *
 * the dense layer's gradients at the active rows (rows are independent).
 *   S [n_rows][Cin], W [Cin][Cout], Y = the layer's output [n_rows][Cout]
 *   (read only with SHC_ACT_RELU), dY [n_rows][Cout]: all of `dtype`;
 *   dS [n_rows][Cin] `dtype` out, dW [Cin][Cout] fp32 out, db [Cout] fp32 out;
 *   each output may be NULL (not computed).
 *   ws: device workspace of shc_sparse_linear_backward_workspace bytes.
 * Every sum has a fixed order: dS in fp32 over Cout, rounded once; dW in
 * fp32 over chunks of rows, the chunks combined in fp64; db in fp32 over
 * splits of rows, combined in fp64.  Results repeat bit for bit on one
 * device (the chunks of the bf16 layer with Cin, Cout in {64, 128}, which
 * runs in one pass over the rows, are sized by the device's CU count).
 * dtype SHC_BF16 or SHC_F32; Cout <= 256.
 */
size_t shc_sparse_linear_backward_workspace(int64_t n_rows, int32_t Cin, int32_t Cout,
                                            int32_t dtype);
int shc_sparse_linear_backward(const void* S, const void* W, const void* Y, const void* dY,
                               int64_t n_rows, int32_t Cin, int32_t Cout, int32_t dtype,
                               int32_t act, void* dS, float* dW, float* db, void* ws,
                               size_t ws_bytes, hipStream_t stream);

/*
 * Slot pair lists of an active set, for the weight gradient of the sparse
 * convolution: every (slot j, row i) with table[j][i] >= 0, slot-major with
 * rows ascending, as int32 pairs[t][2] = (j, i), and pair_ptr[K + 1] with
 * slot j's pairs at [pair_ptr[j], pair_ptr[j + 1]).  table [K][n_rows] from
 * shc_build_neighbor_table; pairs capacity K * n_rows pairs.  Built once per
 * active set and shared by every conv layer on it.
 * ws: device workspace of shc_build_slot_pairs_workspace bytes.
 */
size_t shc_build_slot_pairs_workspace(int64_t n_rows, int32_t K);
int shc_build_slot_pairs(const int32_t* table, int64_t n_rows, int32_t K, int32_t* pairs,
                         int32_t* pair_ptr, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Gradients of the sparse neighbourhood convolution (Eqs. 4-5, Eq. 10),
 * i.e. of the dense convolution of x (.) m restricted to the active rows:
 *
 *   dZ = dY (.) [Y > 0] (SHC_ACT_RELU) or dY,
 *   dW[j] = sum over rows i with table[j][i] >= 0 of S[table[j][i]]^T dZ[i],
 *   db = sum over rows of dZ,
 *   dS[r] = sum over (i, j) with table[j][i] = r of dZ[i] W[j]^T.
 *
 *   S [n_rows][Cin], W [K][Cin][Cout], Y, dY [n_rows][Cout]: all of `dtype`;
 *   table [K][n_rows]: shc_build_neighbor_table of the active set;
 *   pairs, pair_ptr: shc_build_slot_pairs of the same table, or both NULL
 *     (then built inside the call, in the workspace);
 *   table_t, row_slots: shc_build_transposed_table of the same active set;
 *   slot_of, Kt: shc_transpose_neighbors of the mesh;
 *   dS [n_rows][Cin] `dtype` out, dW [K][Cin][Cout] fp32 out, db [Cout] fp32
 *   out; each may be NULL (table_t, row_slots and slot_of are then only read
 *   when dS is requested).
 *   ws: device workspace of shc_sparse_neighbor_conv_backward_workspace bytes.
 * dS sums its terms in ascending virtual slot order in fp32 and rounds once;
 * dW and db as in shc_sparse_linear_backward.  dtype SHC_BF16 or SHC_F32;
 * K <= 32; Cout <= 256.
 */
size_t shc_sparse_neighbor_conv_backward_workspace(int64_t n_rows, int32_t K, int32_t Cin,
                                                   int32_t Cout, int32_t dtype);
int shc_sparse_neighbor_conv_backward(const void* S, const int32_t* table, const int32_t* pairs,
                                      const int32_t* pair_ptr, const int32_t* table_t,
                                      const uint64_t* row_slots, const int32_t* slot_of,
                                      int32_t Kt, const void* W, const void* Y, const void* dY,
                                      int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout,
                                      int32_t dtype, int32_t act, void* dS, float* dW, float* db,
                                      void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Stream-ordering events -- a runtime helper, not an operator of the paper.
 *
 * An event orders work between streams of one device and lets the host wait
 * for that work, like a HIP event made with hipEventDisableTiming, except that
 * its record carries no system-scope fence.  A default HIP event's record
 * writes back and invalidates the device caches for the host's sake; between
 * two streams of one device that costs the stream microseconds per record.
 * Work enqueued after a wait on this event sees every device-memory write of
 * the work recorded before it (a device-scope release and acquire).  The host
 * learns only that the work has finished: its writes to host-visible memory
 * need not be visible to the host yet when shc_event_synchronize returns.
 *
 * shc_event_create      -- *event receives a new event of the current device;
 *                          the caller releases it with shc_event_destroy.
 * shc_event_record      -- records the event on stream: it completes when the
 *                          work enqueued on stream before the record has
 *                          finished.  A new record replaces the last one.
 * shc_stream_wait_event -- work enqueued on stream after this call starts
 *                          only after the event's last record has completed
 *                          (at once if it was never recorded).
 * shc_event_synchronize -- the host waits until the last record has completed.
 * shc_event_destroy     -- releases the event; NULL is accepted and ignored.
 * A NULL event is SHC_ERR_INVALID_ARG (except for destroy); runtime failures
 * are SHC_ERR_HIP.
 */
int shc_event_create(void** event);
int shc_event_record(void* event, hipStream_t stream);
int shc_stream_wait_event(hipStream_t stream, void* event);
int shc_event_synchronize(void* event);
int shc_event_destroy(void* event);

/* ------------------------------------------------------------------------ */
/* Stack executor: the whole path over consecutive batches from native code  */
/* ------------------------------------------------------------------------ */

/*
 * A stack is the path of Sec. 3.2 applied to one batch after another: the
 * mask of a batch is compacted once (Eq. 2, with the neighbour-row table of
 * the active set when a conv layer reads it), and because the active set is
 * the same for every layer (C'_k = C_k), its N' rows run through every layer
 * (Eq. 6 linear or Eqs. 4-5 conv, each with the activation of Eq. 10)
 * before the last layer's rows are scattered back to the dense layout (the
 * zero-filled y (.) m, by shc_scatter or by shc_scatter_update from the
 * previous batch's output) and/or max-pooled per body.  shc_stack_run issues
 * exactly the calls of this header that a caller would issue for the same
 * work, in the same order per stream, from a native loop: results are
 * bit-identical to those calls'.
 *
 * The caller owns every buffer (device memory unless marked host) and
 * describes them once in an shc_stack_desc; shc_stack_create copies the
 * description, checks it and creates the executor's stream-ordering events
 * (device-scope, like shc_event_create's) on the current device.  Buffers
 * must stay allocated until shc_stack_destroy.
 *
 * Streams: with side and tail both NULL the stack is serial: everything
 * runs on the stream given to shc_stack_run, the compaction of batch k + 1
 * enqueued before the scatter and pool of batch k (so the host learns N'
 * while the stream still has work).  With both set (default-priority
 * streams of the same device, distinct from each other and from the run's
 * stream) it is pipelined: the side stream runs batch k + 1's compaction,
 * table and conv plans beside batch k's layers, and the tail stream runs
 * batch k's scatter and pool beside batch k + 1's layers; the last layer's
 * output then alternates between acts[n_layers] and last_alt (the last
 * batch of a run writes acts[n_layers]), and the index sets rotate over
 * three (the host waits for a set's previous scatter and pool to finish
 * before compacting into it).  At the end of a run the run's stream waits
 * for the other two, so work enqueued on it afterwards sees every output.
 */
#define SHC_STACK_MAX_LAYERS 16
#define SHC_LAYER_LINEAR 0 /* Eq. 6 */
#define SHC_LAYER_CONV 1   /* Eqs. 4-5 */

typedef struct shc_stack_layer {
  int32_t kind;      /* SHC_LAYER_LINEAR or SHC_LAYER_CONV */
  int32_t Cin, Cout; /* channels (Cin of layer l = Cout of layer l - 1) */
  int32_t act;       /* SHC_ACT_* */
  const void* W;     /* [Cin][Cout] (linear) or [K][Cin][Cout] (conv), dtype */
  const float* bias; /* [Cout] fp32, or NULL */
  int64_t plan_rows; /* conv: read plan[l] of the index set when 0 < N' <= plan_rows
                        (at most shc_conv_plan_max_rows of the shape); 0: never */
  int64_t split_rows; /* conv: shc_sparse_neighbor_conv_split, with the description's
                         split workspace, when 0 < N' <= split_rows; 0: never.  A layer
                         takes a plan or the split conv, not both. */
  const void* Wp;     /* conv: W packed by shc_pack_conv_weights, or NULL */
  int64_t packed_rows; /* conv: shc_sparse_neighbor_conv_packed with Wp when
                          max(1, packed_min_rows) <= N' <= packed_rows; 0: never.
                          Excludes a plan and the split conv. */
  int64_t packed_min_rows;
} shc_stack_layer;

typedef struct shc_stack_index_set {
  int32_t* coords;      /* [B*V][2] */
  int32_t* inv;         /* [B*V] */
  int32_t* row_ptr;     /* [B+1] */
  int32_t* n_active;    /* [1] device copy of N' */
  int64_t* host_count;  /* host: page-locked and mapped (receives N') */
  void* ws;             /* compaction workspace (shc_compact_mask_workspace) */
  size_t ws_bytes;
  int32_t* table;       /* [K][B*V] neighbour-row table, or NULL without conv layers */
  void* plan[SHC_STACK_MAX_LAYERS]; /* per conv layer with plan_rows > 0: its plan buffer
                                       (layers of one shape may share one; it is built
                                       once per batch), else NULL */
  size_t plan_bytes[SHC_STACK_MAX_LAYERS];
} shc_stack_index_set;

typedef struct shc_stack_desc {
  int32_t B, V, K;         /* bodies, vertices per body, neighbour slots (0: no conv) */
  int32_t dtype;           /* SHC_F32 or SHC_BF16, every feature buffer and weight */
  int32_t C0;              /* input channels = layers[0].Cin */
  const uint8_t* mask;     /* [B*V], read by each batch's compaction */
  const void* x;           /* [B*V][C0] dense input features */
  const int32_t* nbr;      /* [V][K] neighbour lists (conv layers), else NULL */
  int32_t table_in_compaction; /* 1: the compaction writes the table
                                  (shc_compact_mask_table_start), else a
                                  shc_build_neighbor_table call after it */
  int32_t n_layers;        /* 1 .. SHC_STACK_MAX_LAYERS */
  shc_stack_layer layers[SHC_STACK_MAX_LAYERS];
  void* acts[SHC_STACK_MAX_LAYERS + 1]; /* acts[0]: gathered input rows [B*V][C0]
                                           (unused, may be NULL, when layer 0 is linear:
                                           the gather is fused into it); acts[l + 1]:
                                           layer l's output rows [B*V][Cout] */
  void* last_alt;          /* pipelined: second buffer of the last layer's output */
  void* dense_out;         /* [B*V][C_last] scatter output, or NULL for none */
  int32_t incremental;     /* 1: shc_scatter_update from the previous batch's output
                              (dense_out then holds the last scattered batch's y (.) m
                              between runs and is written by nothing else) */
  int32_t* prev_coords;    /* incremental: [B*V][2], the last scattered batch's coords */
  void* pooled;            /* [B][C_last] per-body max-pool output, or NULL for none */
  float pool_empty;        /* pooled value of a body without active rows */
  int32_t n_sets;          /* index sets: 2 (serial) or 3 (pipelined) */
  shc_stack_index_set sets[3];
  hipStream_t side, tail;  /* both NULL (serial) or both set (pipelined) */
  void* split_ws;          /* workspace of the layers with split_rows > 0, at least
                              shc_conv_split_workspace_bytes of each at its split_rows
                              (the layers run one after another and share it), else NULL */
  size_t split_ws_bytes;
} shc_stack_desc;

/* Batch-input callback of shc_stack_run: called just before the compaction
 * of batch `batch` (0-based within the run) is enqueued; it may write that
 * batch's mask and x with work on `stream` (in a pipelined run the side
 * stream, ordered after the gather of batch - 1; the run's stream
 * otherwise).  A nonzero return ends the run with SHC_ERR_INVALID_ARG. */
typedef int (*shc_stack_feed_fn)(void* user, int64_t batch, hipStream_t stream);

/*
 * shc_stack_create  -- *stack receives a new executor for `desc` (copied).
 *   SHC_ERR_INVALID_ARG / _MISALIGNED / _UNSUPPORTED for a description the
 *   calls above would refuse (checked here so that a run does not stop
 *   half-way), SHC_ERR_HIP if an event cannot be created.
 * shc_stack_run     -- `steps` batches on `stream` (and the side and tail
 *   streams).  *cur_set (in/out) is the index set the first batch compacts
 *   into and, on return, the set of the last batch; *prev_rows (in/out,
 *   incremental scatter) the row count of the batch dense_out holds (0 for a
 *   dense_out of zeros).  *n_last receives the last batch's N'.
 *   time_events (may be NULL): 2 * steps caller-owned events, a pair per
 *   batch, recorded on `stream` just before and just after layer time_layer
 *   of that batch (NULL entries: none for that batch).  Returns the first
 *   failing call's status; work enqueued before it stays enqueued (the caller
 *   synchronises the streams before reusing the buffers).  Only one run at a
 *   time per executor.
 * shc_stack_destroy -- releases the executor (NULL is ignored); runs that
 *   used it must have finished.
 */
int shc_stack_create(const shc_stack_desc* desc, void** stack);
int shc_stack_run(void* stack, int64_t steps, hipStream_t stream, shc_stack_feed_fn feed,
                  void* user, int32_t time_layer, void* const* time_events, int32_t* cur_set,
                  int64_t* prev_rows, int64_t* n_last);
int shc_stack_destroy(void* stack);

#ifdef __cplusplus
}
#endif

#endif /* SHC_H_ */
