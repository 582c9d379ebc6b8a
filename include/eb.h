/*
 * eb.h — C ABI of libeb: the jagged, pooled EmbeddingBag forward on one
 * AMD Instinct MI355X (gfx950), with its backward and fused row-wise
 * optimizer step, the un-pooled (sequence) lookup, and the
 * factorization-machine cross term over the pooled output.
 *
 * The operation.  The paper's DLRM study (Sec. IV-A.2, icicle view) splits a
 * recommendation model into sparse_arch, which looks rows up in embedding
 * tables and produces one output embedding per example and categorical
 * feature, and the dense, interaction and over modules that consume them.  The
 * inputs of sparse_arch are jagged categorical features (Abstract; Sec. IV-A.3
 * names embedding-bag lookups over jagged inputs as what sets these models
 * apart from a GEMM-bound LLM), and the stage is bound by memory bandwidth
 * (Sec. IV-A.2).  This library computes exactly that stage:
 *
 *   T tables; table t has R_t rows of D_t elements.  The batch has B examples.
 *   Bag g = t*B + b (table-major) holds the index positions
 *   I_g = [offsets[g], offsets[g+1]).  With x(t,r,d) the fp32 value of element
 *   d of row r of table t (see eb_table_dtype) and w_i the per-sample weight
 *   (1 when no weights are given):
 *
 *     S[d]                      = sum_{i in I_g} w_i * x(t, indices[i], d)
 *     out[b, Doff[t] + d]       = S[d]                   (EB_POOL_SUM)
 *                               = S[d] / |I_g|           (EB_POOL_MEAN)
 *     an empty bag (|I_g| = 0) yields +0.0 in every mode,
 *
 *   where Doff[t] = D_0 + ... + D_{t-1}, so out is [B, sum_t D_t] with the
 *   tables' pooled vectors concatenated in table order.  Sums accumulate in
 *   fp32 starting from +0.0; a bag of one row returns that row's value
 *   (times its weight) rounded once, bit for bit.
 *
 * Memory and ownership.  Every data pointer passed to this library (table
 * rows, indices, offsets, weights, out) is DEVICE memory owned by the caller
 * and must stay valid until the work that uses it has finished on the
 * handle's stream.  The handle copies the table descriptors (not the rows)
 * into a device array that it owns, which also holds the long-bag queue
 * (below).
 *
 * Streams and synchronisation.  The HIP stream is fixed when the handle is
 * created.  eb_forward only enqueues its kernels (per storage type present,
 * the lookup and the long-bag pass below) on it and returns; `out` is valid
 * once that stream has been synchronised.  The other entry points behave the
 * same way.  The handle's tables and settings are fixed at creation; its one
 * piece of mutable device state, the long-bag queue, is used by a lookup and
 * the pass right after it, which each call enqueues under a lock held by the
 * handle, so forwards from several host threads may share it.  eb_forward,
 * eb_forward_fm and eb_forward_seq allocate nothing and, outside checked
 * mode, enqueue only kernel launches, so they may be captured into a HIP
 * graph on the handle's stream and replayed (the captured launches read
 * whatever the buffers hold at replay time; the long-bag pass leaves the
 * queue's counters cleared for the next call, captured or not).  Replay such
 * a graph on the handle's stream, or order it with that stream: two calls on
 * one handle whose kernels run at the same time race on its queue.
 *
 * Long bags (Abstract, Sec. IV-A.3: jagged inputs with long-tailed bag
 * lengths).  A bag of more than 1024 lookups would keep one wavefront busy
 * long after the others, so the wavefront that holds it queues it instead, in
 * segments of 2048 positions, and a second kernel (the long-bag pass) pools
 * the segments on many workgroups: each stages a segment's indices (and
 * weights) in LDS and splits it over four wavefronts; the segments' partial
 * sums are added in segment order, so the result is deterministic (its
 * summation order differs from the one-wavefront order, within the same
 * error bound).  On MI355X a bag of a million lookups takes 0.13 ms so,
 * against 30 ms on one wavefront.  The second kernel costs a few
 * microseconds per call even when no bag is long (1.7-6 us on MI355X), so
 * by default it runs only for batches of
 * at least 2^23 lookups (numel(indices) >= 8388608), where that is under 1%
 * of the lookup, and for batches of at least 64 lookups per bag on average
 * (numel(indices) >= 64 * T * B), which are the ones that hold bags of
 * thousands; EB_LONG_BAG (below) turns it on for every batch.  The queue
 * lives in the handle: up to 16384 segments per call with one partial row of
 * the widest table each (at most 64 MiB; 8 MiB for rows of 128 values); the
 * bags whose segments do not fit are pooled by their own wavefront.  With no
 * long bag the pass's workgroups find the queue empty and exit.
 *
 * Errors.  Every error the host can detect from the arguments is returned
 * before anything is enqueued, and `out` is left untouched.  The kernel never
 * reads outside the tables, indices, offsets or weights, whatever their
 * contents: an index outside [0, R_t) contributes nothing, and offsets are
 * clamped into [0, numel(indices)] and made non-decreasing.  Such inputs
 * break the contract, so the output for the affected bags is unspecified,
 * unless checked mode is on: with the environment variable EB_CHECK=1 set
 * when the handle is created, eb_forward synchronises the stream after the
 * kernel and returns EB_ERR_INDEX_OOB or EB_ERR_OFFSETS if the kernel met
 * such data (offsets[0] != 0 and offsets[T*B] != numel(indices) included).
 * Checked mode is for debugging; it blocks the calling thread.
 *
 * Tuning.  EB_BAGS_PER_WAVE=k (1..32), read when a handle is created, fixes
 * how many consecutive bags of one table a wavefront pools (and how many
 * 64-position chunks a wavefront of eb_forward_seq copies); without it the
 * count is chosen per call from the number of bags (positions).  With 3 or
 * more bags per wavefront, each table's last bags go in short runs that the
 * GPU starts last; EB_TAIL_BAGS=n (n >= 0, 0: none) fixes how many bags of
 * each table that tail holds and EB_TAIL_RUN=r (1..32, default 1) the bags
 * per tail run.  EB_XCD_REMAP=0|1, read
 * at the same time, forces how workgroups map onto the GPU's XCDs (default:
 * XCD-contiguous for handles of up to 32 tables, round-robin otherwise).
 * EB_BWD_TILE_CHUNKS=c (1..16) fixes the backward's tiles at 64*c sorted
 * positions (default: 64, or 128 from about two million lookups on), and
 * EB_BWD_XCD_REMAP=0|1 its workgroup order (default as for the forward);
 * EB_BWD_SORT_ITEMS=4|8|12|16 fixes the backward sort's blocks at 512
 * threads of that many elements (default: chosen per call from the number of
 * lookups and how many of the sort's workgroups the GPU holds at once).
 * EB_LONG_BAG=n (n > 0) runs the long-bag pass for every batch, for bags of
 * more than n lookups (without it: n = 1024, for the batches above);
 * EB_LONG_BAG=0 turns the pass off (every bag is pooled by one wavefront,
 * no second kernel, no queue).  EB_LONG_SEG=s (a
 * power of two from 64 to 2048, default 2048) sets the positions per segment.
 * Results do not depend on any of these, except that the long-bag pass
 * changes the order of a long bag's sum (within the same error bound).
 */
#ifndef EB_H_
#define EB_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EB_OK = 0,
  EB_ERR_INVALID_ARG = -1, /* null pointer, bad count, weights with MEAN ... */
  EB_ERR_DTYPE = -2,       /* unknown table dtype or element type, or a mismatch */
  EB_ERR_SHAPE = -3,       /* sizes that do not fit together */
  EB_ERR_UNSUPPORTED = -4, /* valid request outside what the kernels handle */
  EB_ERR_INDEX_OOB = -5,   /* checked mode: an index outside its table */
  EB_ERR_OFFSETS = -6,     /* checked mode: offsets not a valid partition */
  EB_ERR_OOM = -7,         /* device allocation failed in eb_create_tables */
  EB_ERR_HIP = -8          /* any other HIP runtime error (no device, launch) */
} eb_status;

/*
 * Storage format of one table's rows (row r starts at data + r*row_stride_bytes).
 *   EB_F32:          D fp32 values; x = the value.
 *   EB_F16:          D IEEE binary16 values; x = the value widened to fp32
 *                    (exact).
 *   EB_INT8_ROWWISE: D unsigned 8-bit codes q[0..D), then an fp16 scale s at
 *                    byte D and an fp16 bias c at byte D+2 (little endian);
 *                    x[d] = fp32(s*q[d] + c) rounded once (s*q is exact in
 *                    fp32, so this equals fmaf(s, q, c)).
 *   EB_INT8_ROWWISE_SPLIT: the same values with the scale and bias stored
 *                    apart from the codes: row r holds its D codes only, and
 *                    the rows' 4-byte (fp16 s, fp16 c) words follow all the
 *                    rows as one block, row r's at
 *                    data + num_rows*row_stride_bytes + 4*r.  The table spans
 *                    num_rows*(row_stride_bytes + 4) bytes.  With D = 128 at a
 *                    128-byte stride each row's codes fill one 128-byte line,
 *                    where the packed 132-byte row always touches two; the
 *                    scale/bias block (4 bytes per row) is small enough to
 *                    stay in the GPU's caches while its table is in use.
 * The int8 layouts store the per-row affine (scale, bias) quantisation whose
 * tables make up the single-GPU share of a sharded model (Sec. III-B.1
 * shrinks tables to fit one GPU); the paper fixes no format.
 */
typedef enum { EB_F32 = 0, EB_F16 = 1, EB_INT8_ROWWISE = 2, EB_INT8_ROWWISE_SPLIT = 3 } eb_table_dtype;

/* Element type of an eb_tensor. */
typedef enum { EB_I32 = 0, EB_I64 = 1, EB_T_F32 = 2 } eb_elem_type;

/* Pooling mode.  A weighted sum is EB_POOL_SUM with per_sample_weights. */
typedef enum { EB_POOL_SUM = 0, EB_POOL_MEAN = 1 } eb_pooling;

/*
 * One embedding table.  Requirements, checked by eb_create_tables:
 *   data != NULL; num_rows in [1, 2^31-1]; dim >= 1;
 *   EB_F32:          dim % 4 == 0,  row_stride_bytes >= 4*dim,  data and
 *                    row_stride_bytes multiples of 16;
 *   EB_F16:          dim % 8 == 0,  row_stride_bytes >= 2*dim,  data and
 *                    row_stride_bytes multiples of 16;
 *   EB_INT8_ROWWISE: dim % 16 == 0, row_stride_bytes >= dim+4, data and
 *                    row_stride_bytes multiples of 4 (dim=128 packs rows at
 *                    132 bytes);
 *   EB_INT8_ROWWISE_SPLIT: dim % 16 == 0, row_stride_bytes >= dim, data and
 *                    row_stride_bytes multiples of 16 (dim=128 at 128 bytes),
 *                    and the scale/bias block after the rows readable too.
 *   dim <= 8192.  Any other value gives EB_ERR_INVALID_ARG, an unknown dtype
 *   EB_ERR_DTYPE, a dim or alignment the kernels cannot take
 *   EB_ERR_UNSUPPORTED.
 */
typedef struct {
  const void *data;         /* pointer to row 0 (memory the device can read) */
  int64_t num_rows;         /* R_t */
  int32_t dim;              /* D_t */
  int32_t dtype;            /* eb_table_dtype */
  int64_t row_stride_bytes; /* bytes from row r to row r+1 */
} eb_table_desc;

/* A flat device array: `numel` elements of type `elem_type` at `data`. */
typedef struct {
  const void *data;
  int64_t numel;
  int32_t elem_type; /* eb_elem_type */
} eb_tensor;

/* Opaque handle: the table set, its device descriptor array and its stream. */
typedef struct eb_tables eb_tables;

/*
 * Create a handle for `num_tables` (1 .. 65535) tables described by `descs`
 * (host array, copied).  `hip_stream` is the hipStream_t every eb_forward on
 * this handle enqueues on (NULL = the device's null stream); the current HIP
 * device at this call is the handle's device.  On success *out receives the
 * handle, which the caller releases with eb_destroy.  Synchronous: allocates
 * one small device array (EB_ERR_OOM if that fails) and copies the
 * descriptors into it.  EB_DEVICE_ALLOC_LIMIT=n, read at this call, caps that
 * array at n bytes (about 33 KiB plus 56 bytes per table): a larger one fails
 * with EB_ERR_OOM as if the device were out of memory (for processes that
 * budget device memory).  Each table's rows must be memory the handle's device
 * can read in place: its own device memory, managed memory or pinned host
 * memory; pageable host memory and another device's memory give
 * EB_ERR_INVALID_ARG.  On error *out is set to NULL.
 * Paper: Sec. IV-A.2 (sparse_arch's embedding tables) and Sec. III-B.1
 * (tables too large for one GPU are shrunk to fit it, so the handle takes
 * tables of any row count that fits in device memory).
 */
eb_status eb_create_tables(const eb_table_desc *descs, int32_t num_tables,
                           void *hip_stream, eb_tables **out);

/*
 * Pooled lookup of one batch of jagged categorical features (the jagged
 * features of the Abstract and Sec. IV-A.3 in, sparse_arch's output
 * embeddings of Sec. IV-A.2 out).
 *   indices: EB_I32 or EB_I64, [N]; table-major (all bags of table 0, then
 *            table 1, ...), each value a row number local to its table.
 *   offsets: same element type as indices, [T*B + 1]; offsets[0] = 0,
 *            non-decreasing, offsets[T*B] = N.  B = (numel - 1) / T must be
 *            an integer >= 1 (else EB_ERR_SHAPE); B <= 2^31-1.
 *   per_sample_weights: data == NULL for none; else EB_T_F32 [N]
 *            (EB_ERR_SHAPE if numel != N); not allowed with EB_POOL_MEAN
 *            (EB_ERR_INVALID_ARG).
 *   pooling: EB_POOL_SUM or EB_POOL_MEAN (mean divides by |I_g|).
 *   out:     EB_T_F32 [B * sum_t D_t], row-major [B, sum_t D_t], 16-byte
 *            aligned (EB_ERR_SHAPE if numel differs, EB_ERR_UNSUPPORTED if
 *            misaligned).  Every element is written.
 * Asynchronous on the handle's stream (see checked mode above); allocates
 * nothing.  N = 0 is valid (all bags empty, out is zero-filled).
 */
eb_status eb_forward(const eb_tables *tables, eb_tensor indices,
                     eb_tensor offsets, eb_tensor per_sample_weights,
                     eb_pooling pooling, eb_tensor out);

/*
 * Un-pooled (sequence) lookup: the embedding of every position, for
 * sequence recommenders (the Introduction names HSTU among the architectures
 * the paper's profiling targets), which consume each position of a jagged
 * feature instead of a pooled sum.  For table t and each position i in
 * [start_t, end_t) = [offsets[t*B], offsets[(t+1)*B]):
 *   out[base_t + (i - start_t) * D_t + d] = x(t, indices[i], d),
 *   base_t = sum_{s<t} (end_s - start_s) * D_s,
 * i.e. table t's positions form a [N_t, D_t] row-major block and the blocks
 * follow in table order ([N, D] when every table has the same D).  x is the
 * element's fp32 value as for eb_forward, so the output is exact (one
 * rounding for int8 row-wise rows).
 *   indices, offsets: as for eb_forward; only the table starts offsets[t*B]
 *            (and offsets[T*B] = N) are read.
 *   out:     EB_T_F32 [sum_t N_t * D_t], 16-byte aligned.  With one D for
 *            every table numel must be N * D (else EB_ERR_SHAPE); otherwise
 *            it must lie in [N * min D, N * max D] (else EB_ERR_SHAPE), and a
 *            numel that does not match the offsets leaves the rows that do
 *            not fit unwritten (reported as EB_ERR_SHAPE in checked mode).
 * Positions whose index is outside its table get zeros (EB_ERR_INDEX_OOB in
 * checked mode).  Asynchronous on the handle's stream; allocates nothing;
 * N = 0 enqueues nothing.
 */
eb_status eb_forward_seq(const eb_tables *tables, eb_tensor indices,
                         eb_tensor offsets, eb_tensor out);

/*
 * The factorization-machine cross term of each example over its pooled
 * embeddings.  The DeepFM-based DLRM of the paper feeds sparse_arch's pooled
 * embeddings to inter_arch.fm, which computes the FM cross term (Sec. IV-A.2,
 * inter_arch zoom-in); with field f (table f) of example b represented by its
 * pooled embedding e_{b,f} (the FM second-order term over fields, Rendle 2010):
 *   fm_out[b] = sum_{f < f'} <e_{b,f}, e_{b,f'}>
 *             = 1/2 sum_d [ (sum_f e_{b,f,d})^2 - sum_f e_{b,f,d}^2 ]
 * evaluated in fp32 in one pass over the pooled values (each read once).  The
 * result does not depend on thread scheduling; a handle with one table gives
 * exactly +0.0.  Every table of the handle must have the same dim (else
 * EB_ERR_SHAPE); storage types may differ.
 *   pooled:  EB_T_F32 [B * T * D], row-major [B, T*D] as eb_forward writes it,
 *            16-byte aligned; B = numel / (T*D) must be an integer >= 1
 *            (else EB_ERR_SHAPE).
 *   fm_out:  EB_T_F32 [B], 4-byte aligned (EB_ERR_SHAPE if numel != B,
 *            EB_ERR_INVALID_ARG if NULL).  Every element is written.
 * Asynchronous on the handle's stream; allocates nothing.
 */
eb_status eb_fm_cross(const eb_tables *tables, eb_tensor pooled, eb_tensor fm_out);

/*
 * eb_forward followed by eb_fm_cross on its output, on the handle's stream.
 * out receives exactly what eb_forward writes; fm_out is as for eb_fm_cross.
 * Checked mode as for eb_forward.  Argument errors are those of both calls.
 */
eb_status eb_forward_fm(const eb_tables *tables, eb_tensor indices,
                        eb_tensor offsets, eb_tensor per_sample_weights,
                        eb_pooling pooling, eb_tensor out, eb_tensor fm_out);

/*
 * Training: backward of eb_forward with a fused row-wise optimizer update.
 *
 * The paper profiles each submodule's forward and backward pass (Sec. III-A).
 * For the pooled lookup the gradient of row r of table t is
 *   G[d] = sum over positions i of table t with indices[i] = r of
 *          c_i * grad_out[b(i), Doff[t] + d],
 * c_i = 1 (sum), w_i (weighted sum) or 1/|I_g| (mean), and the rows that
 * occur in the batch are updated in place (the others are left alone):
 *   EB_OPT_SGD:              W[r] -= lr * G
 *   EB_OPT_ROWWISE_ADAGRAD:  s[r] += (1/D) sum_d G[d]^2;
 *                            W[r] -= lr * G / (sqrt(s[r]) + eps)
 * computed in fp32 and rounded once to the table's storage type.  The result
 * does not depend on thread scheduling (no floating-point atomics).
 */
typedef enum { EB_OPT_SGD = 0, EB_OPT_ROWWISE_ADAGRAD = 1 } eb_optimizer;

/*
 * Device workspace (bytes) eb_backward_update needs for num_indices lookups
 * on this handle: 20 bytes per lookup (the sort's two 8-byte element buffers
 * and a bag id), then per tile of 64 or 128 sorted lookups (64*c under
 * EB_BWD_TILE_CHUNKS=c) an 8-byte descriptor and two partial rows of the
 * widest table (8 * max dim bytes), and the sort's counters: 4 bytes per
 * table, pass and digit value, and 8 bytes per pass, digit value and block of
 * 2048 lookups (one more block per table), with digits of up to 9 bits and
 * as many passes as the largest table's row count needs.  Synchronous, host
 * only.
 */
eb_status eb_backward_workspace_size(const eb_tables *tables, int64_t num_indices, size_t *bytes);

/*
 * indices, offsets, per_sample_weights, pooling: as for eb_forward (the batch
 * whose output gradient is grad_out).
 *   grad_out:        EB_T_F32 [B * sum_t D_t], 16-byte aligned, row-major
 *                    [B, sum_t D_t] (the gradient of eb_forward's out).
 *   optimizer:       eb_optimizer; learning_rate, eps as above (eps unused by
 *                    SGD).
 *   optimizer_state: EB_OPT_ROWWISE_ADAGRAD: EB_T_F32 [sum_t R_t], table t's
 *                    rows starting at sum_{s<t} R_s, updated in place;
 *                    ignored by SGD (data may be NULL).
 *   workspace:       device memory of at least eb_backward_workspace_size()
 *                    bytes, 256-byte aligned, owned by the caller; its
 *                    contents are scratch.
 * The tables' rows (the descriptors' data) are written in place.  Only fp32
 * and fp16 tables with dim <= 256 train (else EB_ERR_UNSUPPORTED), and the
 * handle's total row count plus its table count must stay below 2^32.
 * Asynchronous on the handle's stream (checked mode as for eb_forward;
 * there EB_ERR_HIP also reports a sort pass whose bounded wait for an earlier
 * block's counts ran out, which leaves the update wrong but cannot hang);
 * allocates nothing.  Forwards and backwards on one handle are ordered by
 * the stream; two backwards that update the same rows must not overlap.
 */
eb_status eb_backward_update(const eb_tables *tables, eb_tensor indices, eb_tensor offsets,
                             eb_tensor per_sample_weights, eb_pooling pooling, eb_tensor grad_out,
                             int32_t optimizer, float learning_rate, float eps,
                             eb_tensor optimizer_state, void *workspace, size_t workspace_bytes);

/*
 * eb_backward_update for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same computation and arguments without the workspace,
 * which comes from a static device array of EB_NOALLOC_SCRATCH_BYTES bytes
 * (128 MiB) that the library holds on every GPU it runs on until the process
 * ends.  The call allocates nothing and calls no allocating routine.  The
 * workspace this call needs (eb_backward_workspace_size for its lookup
 * count) must fit in the array, else EB_ERR_UNSUPPORTED is returned before
 * anything is enqueued (a batch of about three million lookups into tables
 * of 128-element rows fits).  Every call on one GPU shares that GPU's
 * array: calls that overlap on one GPU (several streams, several host
 * threads) race and must not be issued; calls ordered on one stream are
 * safe.  No part of the array
 * must start at zero, so the contents a previous call left behind are
 * harmless.  EB_ERR_HIP if the array's device address cannot be obtained.
 */
#define EB_NOALLOC_SCRATCH_BYTES 134217728
eb_status eb_backward_update_noalloc(const eb_tables *tables, eb_tensor indices, eb_tensor offsets,
                                     eb_tensor per_sample_weights, eb_pooling pooling, eb_tensor grad_out,
                                     int32_t optimizer, float learning_rate, float eps,
                                     eb_tensor optimizer_state);

/*
 * Release a handle: synchronises its stream, then frees the device array
 * that eb_create_tables allocated and the handle itself (never the tables'
 * rows, which the caller owns).  NULL is a no-op returning EB_OK.  Returns
 * EB_ERR_HIP if the synchronisation or the free fails; the handle is released
 * either way and must not be used again.
 * Handle plumbing of the lookup's life cycle (create, use, destroy); it
 * computes nothing the paper describes.
 */
eb_status eb_destroy(eb_tables *tables);

/*
 * Static, never-NULL English description of a status code (unknown codes
 * give "unknown status").  Host only, thread-safe.
 * Error-reporting plumbing of this interface; no paper passage defines it.
 */
const char *eb_status_string(eb_status s);

#ifdef __cplusplus
}
#endif

#endif /* EB_H_ */
