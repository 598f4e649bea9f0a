/*
 * ssn.h -- C ABI of the MI355X (gfx950) subspace-network stage-boundary codec.
 *
 * The operations follow section 4.1 of the paper ("Pipeline-Parallel
 * Communication with Reparameterized SSNs").  A pipeline stage sends, per
 * token, the k coordinates of its residual-stream activation in a fixed
 * orthonormal basis U (d x k) after subtracting the fixed token embedding
 * E[ids] that both sides of the boundary hold (Eq. (2)); the receiver rebuilds
 * the activation with U^T; gradients travel back through the same projection;
 * and the original SSN re-projects its full-width output projections into
 * span(U) after every optimizer step.  The data-parallel side (section 4.2)
 * adds the per-GPU steps of sparse weight averaging with the delta rule.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensor pointers are DEVICE pointers (hipMalloc / torch CUDA memory),
 *    row-major and contiguous.  The caller owns every buffer; the library
 *    allocates no device memory and keeps no state between calls.
 *  - `dtype` (ssn_dtype_t) is the storage type of X, E, U, G, W and of the
 *    decompressed output.  Coordinates Z and projected gradients G_Z are always
 *    float32 (the paper counts boundary activations in FP32).  All arithmetic
 *    accumulates in float32; bf16 results are rounded to nearest-even once.
 *  - ids are int32 in [0, V).  Ids outside that range are a contract
 *    violation: the kernels clamp them into range (so memory stays in bounds)
 *    and the corresponding output rows are unspecified.
 *  - Every call only enqueues work on `stream` (a hipStream_t; NULL is the
 *    default stream) and returns once the launch is accepted.  Device faults
 *    surface at the caller's next synchronisation.
 *  - Host-side validation runs before any HIP call.  A call with N == 0 (or
 *    n == 0) is a valid no-op that touches no pointer.
 *  - Outputs must not overlap inputs (SSN_ERR_ALIAS), except W, which is
 *    updated in place.  Concurrent calls on different streams are safe.
 *  - Every pointer must be aligned to its element size (SSN_ERR_ALIGN); the
 *    fast paths additionally use 16-byte vector accesses when rows allow it.
 */
#ifndef SSN_H_
#define SSN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SSN_ABI_VERSION 3
/* Largest matrix count accepted by ssn_project_weights_batched. */
#define SSN_MAX_BATCH 16
/* Largest sender count accepted by ssn_sparta_average. */
#define SSN_SPARTA_MAX_SENDERS 64

typedef enum { SSN_F32 = 0, SSN_BF16 = 1 } ssn_dtype_t;

typedef enum {
  SSN_OK = 0,
  SSN_ERR_NULL = 1,        /* a required pointer is NULL                      */
  SSN_ERR_SHAPE = 2,       /* a size is out of range (negative, k > d, ...)  */
  SSN_ERR_DTYPE = 3,       /* unknown dtype                                   */
  SSN_ERR_ALIGN = 4,       /* pointer not aligned to its element size         */
  SSN_ERR_UNSUPPORTED = 5, /* a shape no kernel handles (see each entry)      */
  SSN_ERR_LAUNCH = 6,      /* the HIP launch failed (hipGetLastError)         */
  SSN_ERR_ALIAS = 7        /* an output overlaps an input                     */
} ssn_status_t;

typedef enum {
  SSN_OP_COMPRESS = 0,
  SSN_OP_DECOMPRESS = 1,
  SSN_OP_PROJECT_GRAD = 2,
  SSN_OP_PROJECT_WEIGHTS = 3,
  SSN_OP_COMPRESS_PROJECTED = 4
} ssn_op_t;

/* Returns SSN_ABI_VERSION. */
int ssn_abi_version(void);

/* Static, human-readable name of a status code (never NULL). */
const char *ssn_status_string(int status);

/*
 * Name of the kernel family ("mfma" or "generic") that `op` uses for this
 * dtype and shape when every pointer is 16-byte aligned; "invalid" for an
 * unknown op.  Pure host function (no HIP call), for tests and reports.
 * The MFMA kernels cover bf16 with k <= 128 and: compress / project_grad /
 * compress_projected / decompress d % 128 == 0; project_weights d % 32 == 0
 * (and, when k % 8 != 0, every n % 8 == 0); and float32 storage for
 * compress / project_grad / compress_projected / decompress with d % 64 == 0
 * and U rows of 1 to 128 floats (k, or ldu of a zero-padded basis), and
 * project_weights with d % 32 == 0, k <= 128 and every n % 4 == 0, on
 * float32 MFMA (float32 products and accumulation).  Everything else runs
 * the generic kernels (fp32 arithmetic, one wavefront per token / one block
 * per column).
 */
const char *ssn_kernel_family(ssn_op_t op, ssn_dtype_t dtype, int64_t d, int64_t k);

/*
 * ssn_compress -- sender side of Eq. (2), section 4.1.
 *   Z[i, :] = (X[i, :] - E[ids[i], :]) . U           for i in [0, N)
 *   X   [N, d]  dtype      activations leaving the stage
 *   ids [N]     int32      token ids of those rows
 *   E   [V, d]  dtype      fixed token-embedding table
 *   U   [d, k]  dtype      orthonormal basis (used as stored)
 *   Z   [N, k]  float32    output coordinates
 * Requires 1 <= k <= d, V >= 1.  The subtraction is distributed over the
 * contraction on the bf16 MFMA path (X.U and E[ids].U accumulate by
 * identical fp32 sequences and are subtracted once); the float32 and generic
 * paths subtract in fp32 first.  On all of them compress(E[ids]) is exactly
 * zero.
 */
ssn_status_t ssn_compress(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                          const void *X, const int32_t *ids, const void *E, const void *U,
                          float *Z, void *stream);

/*
 * ssn_decompress -- receiver side of Eq. (2), section 4.1 (reconstruction
 * with U^T), and the sender-side gradient expansion.
 *   Xout[i, :] = E[ids[i], :] + Z[i, :] . U^T        (E, ids non-NULL)
 *   Xout[i, :] =                Z[i, :] . U^T        (E == ids == NULL)
 *   Z    [N, k] float32     coordinates (or projected gradient G_Z)
 *   ids  [N]    int32 / NULL
 *   E    [V, d] dtype / NULL
 *   U    [d, k] dtype
 *   Xout [N, d] dtype       output, rounded once to dtype
 * With N > 0, passing exactly one of E / ids as NULL is SSN_ERR_NULL (with
 * N == 0 every pointer may be NULL, as for the other entries).  The second form is
 * the chain rule through Eq. (2): the gradient w.r.t. the sender's activation
 * is G_Z U^T.
 */
ssn_status_t ssn_decompress(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                            const float *Z, const int32_t *ids, const void *E, const void *U,
                            void *Xout, void *stream);

/*
 * ssn_check_ids -- the ids contract above, checked on the device: writes to
 * *bad the number of i in [0, N) with ids[i] < 0 or ids[i] >= V.
 *   ids [N] int32, bad: one int64 (device memory) output
 * Section 4.1's receiver gathers E[ids] for every token of a microbatch; a
 * caller that wants out-of-range ids to be an error rather than unspecified
 * rows runs this on the same stream before the codec call and reads *bad
 * after a synchronisation.  One launch of one block; the count is a block
 * reduction written by one thread (no atomics), so *bad needs no clearing,
 * and N == 0 writes 0.  Requires V >= 1; bad must not overlap ids.
 */
ssn_status_t ssn_check_ids(int64_t N, int64_t V, const int32_t *ids, int64_t *bad, void *stream);

/*
 * ssn_project_grad -- backward compression, section 4.1 (gradients cross the
 * boundary through the same projection): the receiver sends G_Z = G . U back.
 *   G  [N, d] dtype      gradient w.r.t. the decompressed activation
 *   U  [d, k] dtype
 *   GZ [N, k] float32    output
 */
ssn_status_t ssn_project_grad(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k,
                              const void *G, const void *U, float *GZ, void *stream);

/*
 * Coordinate dtype on the wire, and a padded basis.  The paper sizes the
 * boundary traffic with activations sent in FP32 (section 3.5.2, its estimate
 * of per-node communication), which the entry points above keep.  These
 * variants add two choices:
 *  - `z_dtype`: the dtype of Z (or GZ), SSN_F32 or SSN_BF16 (half the
 *    message).  Compress / project_grad round each fp32 result once to bf16
 *    (nearest even) as they store it; decompress reads bf16 coordinates,
 *    which are exact in its fp32 arithmetic.
 *  - `ldu` (>= k): the row stride of U in elements.  U is then [d, ldu] with
 *    its first k columns the basis and columns k .. ldu-1 ZERO (a padded copy
 *    made once per basis; the basis is fixed for the run).  With ldu a
 *    multiple of 8 (16 for the fastest paths) the kernels read U with aligned
 *    16-byte loads whatever k is, e.g. k = 51 padded to 64; Z keeps k columns.
 *    ldu == k is the plain layout.
 * With z_dtype == SSN_F32 and ldu == k these are exactly the entry points
 * above.  Z is `void *` [N, k] of z_dtype, aligned to its element size;
 * otherwise the arguments, validation and error codes are those of the entry
 * points above (ldu < k, or ldu > 2^31, is SSN_ERR_SHAPE; U's span for the
 * overlap checks is d * ldu elements).
 */
ssn_status_t ssn_compress_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                             int64_t k, int64_t V, const void *X, const int32_t *ids,
                             const void *E, const void *U, int64_t ldu, void *Z, void *stream);
ssn_status_t ssn_decompress_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                               int64_t k, int64_t V, const void *Z, const int32_t *ids,
                               const void *E, const void *U, int64_t ldu, void *Xout,
                               void *stream);
ssn_status_t ssn_project_grad_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                                 int64_t k, const void *G, const void *U, int64_t ldu, void *GZ,
                                 void *stream);

/*
 * ssn_project_grad_ws -- ssn_project_grad_ex with a caller-owned device
 * workspace, for few tokens (the paper's per-call microbatches of 4096 tokens
 * per coalesced batch, sections 3.3.1 and 5.2).  With few tokens every
 * compute unit owns few rows of G and reads all of U; with the workspace d is
 * split into up to 4 ranges whose partial products (float32) go to the
 * workspace, and a second kernel adds them in range order into GZ.
 *   workspace: device memory of workspace_bytes bytes (any contents),
 *     16-byte aligned, not overlapping G, U or GZ (else SSN_ERR_ALIGN /
 *     SSN_ERR_ALIAS); workspace_bytes > 0 with workspace NULL is
 *     SSN_ERR_NULL.  ssn_project_grad_workspace_bytes(dtype, N, d, k, ldu)
 *     is the size that allows every split; it is 0 for the shapes where the
 *     split does not pay (float32 storage, more than 16384 tokens, or U
 *     below 512 KiB), and there the call is ssn_project_grad_ex.  A smaller
 *     workspace (or NULL with 0 bytes) allows fewer ranges or none.
 *   Calls that share a workspace must not overlap in time.
 * The result is within the projection's accuracy of ssn_project_grad_ex's;
 * the sum over d is grouped by range, so the last bits may differ from it
 * and depend on the number of ranges taken (fixed for a shape, a workspace
 * size and a device).  Repeated calls are bitwise reproducible.
 */
size_t ssn_project_grad_workspace_bytes(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k,
                                        int64_t ldu);
ssn_status_t ssn_project_grad_ws(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N, int64_t d,
                                 int64_t k, const void *G, const void *U, int64_t ldu, void *GZ,
                                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * ssn_pad_basis -- the padded layout of the basis used by the `_ex` entry
 * points above, made once per basis (the basis is fixed for the run):
 *   Up[i, c] = U[i, c] for c < k,  Up[i, c] = 0 for k <= c < ldu
 *   U [d, k] dtype, Up [d, ldu] dtype output (k <= ldu <= 2^31).
 * At the paper's rank k = 51, ldu = 64 lets every kernel read U rows as
 * aligned 16-byte pieces: the Pluralis-8B codec kernels at 4096 tokens take
 * 53 instead of 88 us (MI355X).  Up must not overlap U.  One launch.
 */
ssn_status_t ssn_pad_basis(ssn_dtype_t dtype, int64_t d, int64_t k, int64_t ldu, const void *U,
                           void *Up, void *stream);

/*
 * ssn_project_table -- the fixed token embedding projected onto the basis,
 * once:  P[v, :] = E[v, :] . U  for v in [0, V).
 *   E [V, d] dtype, U [d, k] dtype, P [V, k] float32 output
 * Section 4.1 subtracts the fixed token embedding, which both sides of the
 * boundary hold, before projecting (Eq. (2)).  E and U stay fixed for the
 * run, so by linearity (X - E[ids]) U = X U - (E U)[ids], and E U is a table
 * of V x k floats that can be formed once.  The arithmetic is that of
 * ssn_project_grad over the V rows of E (same kernel, same fp32 sequence).
 * Same validation and error codes as ssn_project_grad with N = V.
 */
ssn_status_t ssn_project_table(ssn_dtype_t dtype, int64_t V, int64_t d, int64_t k,
                               const void *E, const void *U, float *P, void *stream);

/*
 * ssn_compress_projected -- Eq. (2) against the projected table:
 *   Z[i, :] = X[i, :] . U - P[ids[i], :]          for i in [0, N)
 *   X [N, d] dtype, ids [N] int32, P [V, k] float32 from ssn_project_table,
 *   U [d, k] dtype, Z [N, k] float32 output
 * Equal to ssn_compress(X, ids, E, U) up to fp32 rounding when P was made by
 * ssn_project_table from (E, U) with the same dtype, d and k.  A row X[i]
 * equal to E[ids[i]] compresses to zero up to that rounding, and exactly to
 * zero when N and V select the same kernel (both 32768 or more, or both
 * fewer, on 16-byte aligned buffers).  It reads X and k floats of P per token
 * instead of X and d elements of E per token (about half the bytes of
 * ssn_compress at d = 4096, k = 64, bf16).  Validation as ssn_compress, with
 * P in place of E (P must be 4-byte aligned and must not overlap Z).
 */
ssn_status_t ssn_compress_projected(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                                    const void *X, const int32_t *ids, const float *P,
                                    const void *U, float *Z, void *stream);
/* The same with a coordinate dtype and a padded basis (see ssn_compress_ex):
 * the table P stays float32 [V, k]; with SSN_BF16 each Z value is rounded
 * once after the subtraction. */
ssn_status_t ssn_compress_projected_ex(ssn_dtype_t dtype, ssn_dtype_t z_dtype, int64_t N,
                                       int64_t d, int64_t k, int64_t V, const void *X,
                                       const int32_t *ids, const float *P, const void *U,
                                       int64_t ldu, void *Z, void *stream);

/*
 * ssn_project_weights -- original-SSN re-projection after an optimizer step
 * (section 4.1, and section 6.1 which contrasts it with the reparameterized
 * form): the rows of every output projection are pulled back into span(U).
 * With PyTorch's [out = d, in = n] layout this is
 *   W <- U . (U^T . W)        in place, W [d, n] dtype, U [d, k] dtype
 * U^T W is accumulated in fp32 and never leaves the chip; W is read once and
 * written once.  Requires 1 <= k <= d.  k > 1024 is SSN_ERR_UNSUPPORTED.
 * `workspace` (device, caller-owned) holds at least
 * ssn_project_weights_workspace_bytes(d, n, k) bytes, else SSN_ERR_SHAPE; it
 * may be NULL when that size is 0.  The kernels keep the k x n partial
 * product U^T W in registers and LDS of the compute unit that owns those
 * columns (each block reads its whole column strip of W before writing it
 * back), so the size is 0 for every shape today; the argument keeps room for
 * a split of d across blocks, which would stage U^T W in device memory.
 * Matrices wider than 2^31 - 1 columns run the generic kernel.
 */
size_t ssn_project_weights_workspace_bytes(int64_t d, int64_t n, int64_t k);
ssn_status_t ssn_project_weights(ssn_dtype_t dtype, int64_t d, int64_t n, int64_t k,
                                 void *W, const void *U, void *workspace, size_t workspace_bytes,
                                 void *stream);

/*
 * ssn_project_weights_batched -- the same re-projection for `count` matrices
 * that share d and U (e.g. every attention and MLP output projection of a
 * pipeline stage), in one launch.
 *   W[b] [d, n[b]] dtype, in place, for b in [0, count)
 *   W and n are HOST arrays of `count` entries; 1 <= count <= SSN_MAX_BATCH.
 * Matrices must not overlap each other.  With bf16 storage a matrix gets the
 * same bits alone and in a batch.  The float32 kernel splits the sum over d
 * between the waves that share a column tile, and that split follows the
 * column partition of the launch (the total column count and the device's
 * compute units), so there the two may differ in the last bits.
 */
ssn_status_t ssn_project_weights_batched(ssn_dtype_t dtype, int64_t count, int64_t d,
                                         const int64_t *n, int64_t k, void *const *W,
                                         const void *U, void *stream);

/*
 * Reparameterized SSN (section 4.1, Eq. (3)).  An output projection
 * W [din, d] (Eq. (1)'s row-vector convention: a layer adds H W to the
 * residual stream) is trained as its factor Zp [din, k] with W = Zp U^T, so
 * every row of W lies in span(U) by construction and W is never formed.
 *   H  [N, din] dtype   layer input (attention concat or MLP hidden)
 *   Zp [din, k] dtype   trainable factor
 *   U  [d, k]   dtype   the shared basis
 * Shape rules: 1 <= k <= d, k <= din; N == 0 is a no-op (backward: GZp = 0).
 * All intermediate products accumulate in fp32; bf16 outputs are rounded once.
 * Zp and U may be stored with zero columns appended up to a whole number of
 * 16-column tiles (pass the padded width as k): that is the same layer, the
 * padding columns of T, GT and GZp stay zero, and the kernels take their
 * aligned paths (k = 51 padded to 64 at din = 18432, d = 5120, N = 4096:
 * forward and backward 175 -> 155 us on MI355X).
 */

/*
 * ssn_reparam_forward -- the layer's contribution Y = (H Zp) U^T.
 *   T [N, k] float32   output: the projected input H Zp (the backward needs
 *                      only G, H and Zp, but T is what crosses to U^T)
 *   Y [N, d] dtype     output
 * Two launches on `stream` (the projection of H by Zp, then the expansion
 * by U^T), or three when, with few tokens, the projection splits din into
 * up to four ranges: their float32 partial products are staged in Y's
 * memory (before Y is written) and summed in a fixed order.  The number of
 * ranges depends on the shape and the device's compute-unit count.
 * Outputs must not overlap inputs or each other.
 */
ssn_status_t ssn_reparam_forward(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d, int64_t k,
                                 const void *H, const void *Zp, const void *U, float *T, void *Y,
                                 void *stream);

/*
 * Bytes of device workspace ssn_reparam_backward needs for these sizes
 * (partial factor gradients of the token splits; 0 when none is needed).
 * Depends on (dtype, N, din, k) only.
 */
size_t ssn_reparam_workspace_bytes(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t k);

/*
 * ssn_reparam_backward -- gradients of the layer for G = dL/dY [N, d]:
 *   GT  [N, k]   float32  output: G U
 *   GH  [N, din] dtype    output: dL/dH = (G U) Zp^T
 *   GZp [din, k] float32  output: dL/dZp = (dL/dW) U = H^T (G U)
 * `workspace` (device, 4-byte aligned, caller-owned) holds at least
 * ssn_reparam_workspace_bytes(dtype, N, din, k) bytes, else SSN_ERR_SHAPE.
 * The factor gradient is summed over token splits in a fixed order
 * (deterministic).  Like the forward, G U may split d into ranges staged in
 * GH's memory before GH is written.  Three to five launches on `stream`.
 */
ssn_status_t ssn_reparam_backward(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d, int64_t k,
                                  const void *H, const void *Zp, const void *U, const void *G,
                                  float *GT, void *GH, float *GZp, void *workspace,
                                  size_t workspace_bytes, void *stream);

/*
 * ssn_reparam_backward_noalloc -- ssn_reparam_backward for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the same kernels and results, with
 * the factor gradient's partial sums in the library's own scratch array of
 * SSN_NOALLOC_SCRATCH_BYTES per device instead of a caller workspace.  The
 * caller still passes every input and output.  Arguments and errors are those
 * of ssn_reparam_backward; a shape whose ssn_reparam_workspace_bytes exceeds
 * SSN_NOALLOC_SCRATCH_BYTES is SSN_ERR_UNSUPPORTED; none is: the token
 * splits times din never exceed 256 column blocks of 512 (k <= 64) or 256
 * (64 < k <= 128), so the partial sums take at most 32 MiB, and k > 128
 * needs no workspace.  Allocates nothing: the array is part of the library's device
 * code, held by every GPU the library runs on until the process ends; its
 * address is looked up on the first call on each device.  All calls on one
 * GPU share that GPU's array, so calls that overlap in time on one GPU (on
 * different streams, or from several host threads) race and must be ordered
 * by the caller; each call writes every scratch value it reads, so nothing
 * carries over from the previous call.
 */
#define SSN_NOALLOC_SCRATCH_BYTES (32u << 20)
ssn_status_t ssn_reparam_backward_noalloc(ssn_dtype_t dtype, int64_t N, int64_t din, int64_t d,
                                          int64_t k, const void *H, const void *Zp,
                                          const void *U, const void *G, float *GT, void *GH,
                                          float *GZp, void *stream);

/*
 * ssn_factored_embedding -- the trainable embedding factored through the
 * basis, T_S = E U^T (section 4.1), looked up by token id:
 *   X0[i, :] = E[ids[i], :] . U^T
 *   ids [N] int32, E [V, k] float32, U [d, k] dtype, X0 [N, d] dtype output.
 * Same kernel as ssn_decompress (expansion form) with the coordinate rows
 * gathered by id.
 */
ssn_status_t ssn_factored_embedding(ssn_dtype_t dtype, int64_t N, int64_t d, int64_t k, int64_t V,
                                    const int32_t *ids, const float *E, const void *U, void *X0,
                                    void *stream);

/*
 * Sparse weight averaging with the delta rule (section 4.2, Eq. (sparta) and
 * Eq. (delta_rule); the averaging round of the worker in section 3.3.1): the
 * one-GPU steps of a round over the float32 master weights theta [n].  A round
 * selects m positions P (p = 5% of the parameters in the paper):
 *   I != NULL   P_i = I[i], I an int64 DEVICE array of m DISTINCT positions
 *               in [0, n).  Entries outside [0, n) are a contract violation:
 *               they are clamped into range (memory stays in bounds) and the
 *               affected values are unspecified; repeated positions race.
 *   I == NULL   the segment P_i = first + i, with 0 <= first and
 *               first + m <= n (else SSN_ERR_SHAPE).  The paper tiles theta
 *               with 20 such segments and rotates through them.
 * All arithmetic is float32; m == 0 is a no-op.  Segment calls whose pointers
 * are 16-byte aligned (and m % 4 == 0) use 16-byte accesses.
 */

/*
 * ssn_sparta_segment -- the segment averaged in round r: the run shares
 * p = 1/segments of the parameters per round, and consecutive rounds cover
 * every parameter once per `segments` rounds (p = 5 %, 20 rounds in the
 * paper).  Segment s = [floor(s n / S), floor((s + 1) n / S)) for
 * S = segments, and round r averages segment r mod S: the S segments tile
 * [0, n) in order and their sizes differ by at most one.  Host function (no
 * HIP call): writes *first and *m, the arguments of the segment form above.
 * Requires n >= 0, r >= 0, 1 <= segments <= 2^20 (else SSN_ERR_SHAPE) and
 * non-NULL outputs (SSN_ERR_NULL).
 */
ssn_status_t ssn_sparta_segment(int64_t n, int64_t r, int64_t segments, int64_t *first,
                                int64_t *m);

/*
 * ssn_sparta_snapshot -- snap[i] = theta[P_i], the copy each replica takes at
 * the start of a round.  theta [n] float32, snap [m] float32 output; snap
 * must not overlap theta or I.  One launch.
 */
ssn_status_t ssn_sparta_snapshot(int64_t n, int64_t m, const int64_t *I, int64_t first,
                                 const float *theta, float *snap, void *stream);

/*
 * ssn_sparta_average -- the reducer's step for one slice of m values from R
 * senders:
 *   acc[i]      = sum_r w_r chunks[r][i] / sum_r w_r   (senders summed in order)
 *   deltas[r][i] = acc[i] - chunks[r][i]                (what sender r receives)
 * chunks and deltas are HOST arrays of R device pointers ([m] float32 each);
 * weights is a HOST array of R floats, or NULL for all ones.  Weights must be
 * finite and >= 0 with a positive sum (else SSN_ERR_SHAPE); a sender with
 * weight 0 adds nothing to acc and still gets its delta.  deltas may be NULL,
 * and so may any entry (that delta is not written).  1 <= R <=
 * SSN_SPARTA_MAX_SENDERS.  Outputs must not overlap the chunks or each other.
 * One launch.
 */
ssn_status_t ssn_sparta_average(int64_t R, int64_t m, const float *const *chunks,
                                const float *weights, float *acc, float *const *deltas,
                                void *stream);

/*
 * ssn_delta_rule -- apply a finished round to the weights, in place:
 *   theta[P_i] += lambda * (avg[i] - snap[i])
 * avg [m] float32 is the group average, snap [m] float32 the snapshot taken
 * at the start of the round, so progress made meanwhile is kept (the paper
 * uses lambda = 1).  snap may be NULL: theta[P_i] += lambda * avg[i], which
 * is also how a replica adds the delta a reducer returned to its buffer.
 * lambda must be finite (else SSN_ERR_SHAPE).  theta must not overlap avg,
 * snap or I.  One launch.
 */
ssn_status_t ssn_delta_rule(int64_t n, int64_t m, const int64_t *I, int64_t first, float *theta,
                            const float *avg, const float *snap, float lambda, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SSN_H_ */
