/*
 * adapm.h -- C ABI of a single-GPU (MI355X, gfx950) sparse parameter store.
 *
 * The store is the node-local parameter store that a parameter manager
 * provides to its workers: global read and write access to model parameters
 * by key (Section 1), served locally from memory shared with the workers
 * (Section 4, Figure 3), with the updates of all workers to one parameter
 * merged into the store (Appendix B.1.2).  Every task in the paper trains
 * with SGD and AdaGrad (Appendix C); the store applies AdaGrad on write.
 *
 * Semantics of one step (deterministic, synchronous minibatch):
 *   pull all rows the batch needs from the pre-step table, compute
 *   per-occurrence gradients from those values, sum the gradients of each
 *   distinct key, apply one AdaGrad update per distinct key:
 *     G <- G + g*g ;  W <- W - lr * ( g / (sqrt(G) + eps) )    (fp32, per element)
 *   Sums of more than one term are accumulated in fp64 and rounded once.
 *
 * Conventions shared by all calls
 *   - Plain C types only.  "device" pointers are HIP device memory (e.g. a
 *     torch.cuda tensor's data_ptr()); "host" pointers are ordinary memory.
 *   - Tables are fp32, row-major, dense: row k of a table with `dim` columns
 *     starts at element k*dim.  The caller owns the value table W and the
 *     AdaGrad accumulator table G (both num_keys*dim floats, device); the
 *     store borrows them for its lifetime and never frees them.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Every
 *     call is enqueued asynchronously on that stream; nothing synchronizes
 *     unless stated.  A store must be used from one stream at a time.
 *   - Argument errors are detected on the host before anything is enqueued
 *     and returned immediately (nothing is launched).  Errors that only the
 *     device can see (a key outside [0, num_keys)) set a sticky flag in the
 *     store that ps_get_error() reports; the offending pulled row is zero,
 *     and the offending occurrence (or the whole training unit it belongs
 *     to, for the step calls) contributes nothing.
 *   - n = 0 (or B = 0) is a valid no-op that returns PS_OK.
 *   - Output buffers must not alias the tables or each other.
 *   - Workspace: calls that need scratch memory take (ws, ws_bytes) from
 *     the caller, sized by ps_workspace_bytes(); the library allocates no
 *     device memory except a small status block in ps_create() (and, once
 *     per device, the static scratch array of ps_push_noalloc).
 *   - Two-phase calls (the *_prepare / *_apply pairs): the apply trusts the
 *     workspace its prepare filled (sorted keys, permutation, segments,
 *     validity) and does not check it again; an apply on a workspace that
 *     no matching prepare filled, or with other ids than the prepare's, is
 *     undefined behaviour (its kernels index the tables with whatever the
 *     workspace holds).
 */
#ifndef ADAPM_H
#define ADAPM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ps_store ps_store;   /* opaque host handle */
typedef int32_t ps_status;

#define PS_OK               0
#define PS_ERR_INVALID     (-1)   /* bad argument (null pointer, negative size, bad dim ...) */
#define PS_ERR_KEY_RANGE   (-2)   /* a key outside [0, num_keys) was seen on the device */
#define PS_ERR_WORKSPACE   (-3)   /* ws_bytes smaller than ps_workspace_bytes() */
#define PS_ERR_DEVICE      (-4)   /* a HIP runtime call failed */
#define PS_ERR_UNSUPPORTED (-5)   /* a size beyond what the kernels handle */
#define PS_ERR_NOT_RESIDENT (-6)  /* staged store: a key with no slot was accessed */

/* operation codes for ps_workspace_bytes() */
#define PS_OP_PULL      0
#define PS_OP_PUSH      1
#define PS_OP_DEDUP     2
#define PS_OP_STEP_MF   3
#define PS_OP_STEP_KGE  4
#define PS_OP_STEP_SGNS 5
#define PS_OP_STEP_CTR  6
#define PS_OP_STEP_MF_ASYNC 7

/* Limits: num_keys in [1, 2^31-1]; dim in [1, 512]; key occurrences per
 * call n < 2^31 - 2^20.  Stores made by ps_create / ps_create_strided may
 * also hold wider rows, dim in (512, 16384] and a multiple of 4 (the paper's
 * widest models keep 1,000 floats per parameter row, Table 3): ps_pull,
 * ps_push (and its two-phase and allocation-free forms) and ps_dedup serve
 * them, one column slice of 512 floats at a time (per-element AdaGrad and
 * per-element sums do not mix columns, so the result is the whole-row
 * update); the task steps, ps_push_async and ps_step_mf_async return
 * PS_ERR_UNSUPPORTED for them, and row-wise, bf16 and staged stores keep
 * dim <= 512. */

/* Create a store over caller-owned device tables W (values) and G
 * (AdaGrad accumulators), each num_keys*dim floats, with AdaGrad learning
 * rate lr > 0 and eps >= 0.  The store is the node-local parameter store
 * that the workers of a node share (Section 4, Figure 3); every task of
 * Appendix C trains its parameters with AdaGrad.  Allocates one small
 * device status block and clears it on `stream`.  *out receives the handle
 * (NULL on error). */
ps_status ps_create(ps_store** out, int64_t num_keys, int32_t dim, float* values, float* accum,
                    float lr, float eps, void* stream);

/* As ps_create, with a row stride: row k of W starts at values + k*row_stride
 * and row k of G at accum + k*row_stride (row_stride >= dim floats; a
 * multiple of 4 when dim is).  ps_create is the dense case row_stride = dim.
 * One allocation of [num_keys][2*dim] floats with accum = values + dim keeps
 * each key's value and accumulator rows side by side, so an update touches
 * one 8*dim-byte region of HBM instead of two.  Rows of W and G must not
 * overlap (PS_ERR_INVALID otherwise).  Pulled rows are always dense. */
ps_status ps_create_strided(ps_store** out, int64_t num_keys, int32_t dim, int64_t row_stride,
                            float* values, float* accum, float lr, float eps, void* stream);

/* As ps_create_strided, with row-wise AdaGrad: one accumulator per key
 * instead of one per element, an update variant (the paper's tasks use
 * per-element AdaGrad, Appendix C) that halves the update's table traffic.
 * For the merged gradient row g of a key (fp32) and its accumulator a:
 *   a <- a + fp32( (sum_c g_c*g_c) / dim )   (squares and sum in fp64)
 *   W <- W - lr * ( g / (sqrt(a) + eps) )    (fp32, per element, in this order)
 * Merging and all other semantics are those of the per-element store.
 * The accumulator of key k is accum[k*accum_stride] (device, caller-owned,
 * accum_stride >= 1).  It may be a separate vector (accum_stride = 1) or
 * sit in the padding of each value row (accum = values + c with
 * dim <= c < row_stride and accum_stride = row_stride), so that a key's
 * update touches one region of HBM.  An accumulator inside a value row is
 * PS_ERR_INVALID. */
/* As ps_create, with bf16 values: row k of the values is values +
 * k*value_stride (uint16 words, each the upper half of an fp32 word), row k
 * of the fp32 AdaGrad accumulators accum + k*accum_stride: two separate
 * allocations, or rows interleaved in one (equal byte strides, each key's
 * accumulator row after its value row), so that an update touches one
 * span of HBM.  An update variant that halves the bytes of a value: reads
 * widen exactly to fp32, arithmetic and accumulators are unchanged, and the
 * updated value is narrowed once to the nearest bf16 (ties to even).
 * ps_pull returns fp32 rows; ps_push and the MF steps run on such a store;
 * the other steps return PS_ERR_UNSUPPORTED.  When dim % 4 == 0 the values
 * must be 8-byte aligned, the accumulators 16-byte aligned and both strides
 * multiples of 4. */
ps_status ps_create_bf16(ps_store** out, int64_t num_keys, int32_t dim, uint16_t* values, int64_t value_stride,
                         float* accum, int64_t accum_stride, float lr, float eps, void* stream);

ps_status ps_create_rowwise(ps_store** out, int64_t num_keys, int32_t dim, int64_t row_stride,
                            float* values, float* accum, int64_t accum_stride, float lr, float eps,
                            void* stream);

/* Free the handle and its status block (not the tables).  NULL is a no-op.
 * Synchronizes the device before freeing. */
ps_status ps_destroy(ps_store* s);

/* Workspace bytes a call needs.  `units` is the batch size of the call
 * (keys for PULL/PUSH/DEDUP; entries, triples, centres or samples for the
 * steps) and `per_unit` the key occurrences each unit creates: 1 for
 * PULL/PUSH/DEDUP, 2 for MF, 3+n_neg for KGE, 1+2*window*(1+n_neg) for
 * SGNS, F for CTR (2 for MF_ASYNC).  Returns 0 for an invalid
 * combination. */
size_t ps_workspace_bytes(int64_t num_keys, int32_t dim, int32_t op, int64_t units, int64_t per_unit);

/* Read access (Section 1: global read access to parameters by key).
 * out[i*dim + c] = W[keys[i]*dim + c] for i < n, a bit copy.
 * keys: device int64[n]; out: device float[n*dim].  No workspace. */
ps_status ps_pull(ps_store* s, const int64_t* keys, int64_t n, float* out, void* stream);

/* Write access with merging (Appendix B.1.2: updates to a parameter are
 * merged into its store; Appendix C: AdaGrad).  grads[i*dim..] is the
 * gradient row of occurrence i with key keys[i]; all occurrences of one key
 * are summed (fp64, then rounded to fp32) and one AdaGrad update is applied
 * per distinct key.  keys: device int64[n]; grads: device float[n*dim]. */
ps_status ps_push(ps_store* s, const int64_t* keys, int64_t n, const float* grads,
                  void* ws, size_t ws_bytes, void* stream);

/* ps_push in two phases, for callers that overlap the key work of the next
 * push with the merge of this one (two workspaces, two streams), as
 * ps_step_mf_prepare / ps_step_mf_apply do for the MF step.
 * ps_push_prepare reads only the keys and writes the workspace (key
 * intake, sort, segments; a key outside [0, num_keys) raises the store's
 * sticky error here); it reads and writes no table row, so it may run
 * while another workspace's apply updates W and G.  ps_push_apply then
 * merges grads (device float[n*dim], as for ps_push) into W and G in the
 * order that workspace holds; it no longer reads the keys.  ws must hold
 * the result of ps_push_prepare for this store and the same n, unmodified;
 * the order of prepare before apply, and of an apply before the next
 * prepare into the same workspace, is the caller's (e.g. events).
 * Prepare then apply on one stream is exactly ps_push.  Workspace size:
 * ps_workspace_bytes(num_keys, dim, PS_OP_PUSH, n, 1).  Staged stores:
 * PS_ERR_UNSUPPORTED. */
ps_status ps_push_prepare(ps_store* s, const int64_t* keys, int64_t n, void* ws, size_t ws_bytes, void* stream);
ps_status ps_push_apply(ps_store* s, int64_t n, const float* grads, void* ws, size_t ws_bytes, void* stream);

/* ps_push for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same merge and update, with the workspace taken from a static device array
 * of PS_NOALLOC_SCRATCH_BYTES that the library holds, one per device, from
 * the first store created on that device until the process ends.  The call
 * allocates nothing and sets no memory with hipMemset.  A push whose
 * workspace (ps_workspace_bytes(num_keys, dim, PS_OP_PUSH, n, 1)) exceeds
 * the array returns PS_ERR_UNSUPPORTED before anything is enqueued (the
 * limit is about 1,500,000 keys at dim 16, 770,000 at dim 100 and 227,000
 * at dim 512).  Every call on one device
 * shares that device's array and leaves its contents behind, so calls that
 * overlap on one device (other streams, other stores, other threads) race
 * and must be ordered by the caller.  Kernel timing (ps_set_timing) creates
 * events and should be off. */
#define PS_NOALLOC_SCRATCH_BYTES (64u << 20)
ps_status ps_push_noalloc(ps_store* s, const int64_t* keys, int64_t n, const float* grads, void* stream);

/* The merge order used by ps_push (the updates of one parameter are merged
 * before they reach the store, Appendix B.1.2), exposed for bit-exact
 * checking: a stable sort of the occurrences by key.  There is no store,
 * so a device flag `err` takes the place of the store's sticky error.  Keys outside [0, num_keys) sort after all
 * valid keys in their original order and belong to no segment.
 *   uniq      device int64[n]  : distinct valid keys ascending (first U used)
 *   perm      device int32[n]  : occurrence index at each sorted position
 *   offsets   device int32[n+1]: offsets[u] = first sorted position of uniq[u],
 *                                offsets[U] = number of valid occurrences
 *   num_unique device int32[1] : U
 *   err       device int32[1] or NULL: set to 1 if an invalid key was seen
 *                                (never cleared by this call)            */
ps_status ps_dedup(int64_t num_keys, const int64_t* keys, int64_t n, int64_t* uniq, int32_t* perm,
                   int32_t* offsets, int32_t* num_unique, int32_t* err,
                   void* ws, size_t ws_bytes, void* stream);

/* One matrix-factorization step (Appendix C, "Matrix factorization").
 * Entry b = (row[b], col[b], val[b]) uses keys u = row[b] and
 * m = col_key_offset + col[b]; with e = val - <W_u, W_m>:
 *   loss = e^2/2 + lambda/2 (|W_u|^2 + |W_m|^2)
 *   grad_u = lambda W_u - e W_m ,  grad_m = lambda W_m - e W_u
 * row, col: device int32[B]; val: device float[B]; loss: device double[1]
 * receives the summed loss of the step (may be NULL). */
ps_status ps_step_mf(ps_store* s, const int32_t* row, const int32_t* col, const float* val,
                     int64_t B, int64_t col_key_offset, float lambda, double* loss,
                     void* ws, size_t ws_bytes, void* stream);

/* ps_step_mf in two phases, for callers that overlap the key work of the
 * next batch with the table update of this one (two workspaces, two
 * streams).  ps_step_mf_prepare reads only the batch and writes the
 * workspace (sorted keys, segments, one record per entry); it reads no
 * table row, so it may run while another workspace's apply updates W and G.
 * ps_step_mf_apply then updates W and G from that workspace (and writes
 * the loss); it no longer reads row, col or val.  ws must hold the
 * result of ps_step_mf_prepare for this store and the same B, unmodified;
 * ordering prepare before apply (and an apply before the next prepare into
 * the same workspace) is the caller's, e.g. with events.  Prepare then
 * apply on one stream is exactly ps_step_mf.  rows_done (a hipEvent_t, may
 * be NULL) is recorded on the stream once the row-key merge has been
 * enqueued: a prepare that waits for it overlaps the rest of the apply
 * (column-key merge, finalize) instead of the bandwidth-bound row merge. */
ps_status ps_step_mf_prepare(ps_store* s, const int32_t* row, const int32_t* col, const float* val,
                             int64_t B, int64_t col_key_offset, void* ws, size_t ws_bytes, void* stream);
ps_status ps_step_mf_apply(ps_store* s, int64_t B, float lambda, double* loss, void* ws,
                           size_t ws_bytes, void* stream, void* rows_done);

/* Unmerged write access: the asynchronous update semantics of the paper's
 * experiments (Section 5.1, asynchronous SGD), as an opt-in alternative to
 * ps_push.  Every occurrence's gradient row is applied as its own AdaGrad
 * step (per element, or row-wise on a row-wise store), each element update
 * a device-scope atomic add: an occurrence's step uses the accumulator just
 * after its own square was added.  Occurrences of one key are applied in
 * no fixed order, so results are not reproducible bit for bit; element by
 * element they equal those of applying the occurrences one after another
 * in some order.  Needs no sort and no workspace.  keys: device int64[n];
 * grads: device float[n*dim], row-major.  A key
 * outside [0, num_keys) is skipped and reported by ps_get_error.  Staged
 * stores and bf16 values: PS_ERR_UNSUPPORTED. */
ps_status ps_push_async(ps_store* s, const int64_t* keys, int64_t n, const float* grads, void* stream);

/* The MF step of ps_step_mf with the unmerged update: both gradient rows of
 * every entry from the pre-step table (as in ps_step_mf), then applied as
 * by ps_push_async (occurrence 2b: the row key, 2b+1: the column key).  ws
 * holds the 2*B gradient rows: ps_workspace_bytes(num_keys, dim,
 * PS_OP_STEP_MF_ASYNC, B, 2).  loss as for ps_step_mf. */
ps_status ps_step_mf_async(ps_store* s, const int32_t* row, const int32_t* col, const float* val,
                           int64_t B, int64_t col_key_offset, float lambda, double* loss,
                           void* ws, size_t ws_bytes, void* stream);

/* One ComplEx knowledge-graph-embedding step with negative sampling
 * (Appendix C, "Knowledge graph embeddings").  Rows hold [Re | Im] of a
 * complex vector of dim/2 components (dim must be even).  Triple t uses
 * keys head[t], rel_key_offset + rel[t], tail[t]; neg[t*n_neg + j] replaces
 * the head for j < n_head_neg and the tail otherwise.  Score
 * phi = Re(sum_k s_k r_k conj(o_k)); loss softplus(-y phi), y = +1 for the
 * true triple and -1 for each corrupted one.
 * head, rel, tail: device int32[B]; neg: device int32[B*n_neg]. */
ps_status ps_step_kge(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                      const int32_t* neg, int64_t B, int32_t n_neg, int32_t n_head_neg,
                      int64_t rel_key_offset, double* loss, void* ws, size_t ws_bytes,
                      void* stream);

/* ps_step_kge in two phases, as ps_step_ctr_prepare / ps_step_ctr_apply:
 * the prepare reads only the ids (triple validity, key sort, segments into
 * ws; no table row), the apply forms the gradients from the pre-step table,
 * merges them into W and G and writes the loss, reading head, rel, tail and
 * neg again: they must be the arrays given to the prepare, unchanged, with
 * the same B, n_neg and rel_key_offset, and ws that prepare's result,
 * unmodified.  Prepare then apply gives exactly the results of ps_step_kge.
 * Workspace size: ps_workspace_bytes(num_keys, dim, PS_OP_STEP_KGE, B,
 * 3 + n_neg).  Staged stores: PS_ERR_UNSUPPORTED. */
ps_status ps_step_kge_prepare(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                              const int32_t* neg, int64_t B, int32_t n_neg, int64_t rel_key_offset, void* ws,
                              size_t ws_bytes, void* stream);
ps_status ps_step_kge_apply(ps_store* s, const int32_t* head, const int32_t* rel, const int32_t* tail,
                            const int32_t* neg, int64_t B, int32_t n_neg, int32_t n_head_neg, int64_t rel_key_offset,
                            double* loss, void* ws, size_t ws_bytes, void* stream);

/* One skip-gram negative-sampling step (Appendix C, "Word vectors").
 * Centre b has input key centre[b]; slot q < 2*window holds a context word
 * ctx[b*2w + q] (-1 = no word, the slot is skipped) and n_neg negatives
 * neg[(b*2w + q)*n_neg + k]; output keys are out_key_offset + word.  With
 * x = <u, v_centre>: loss softplus(-x) for the context, softplus(x) for a
 * negative; grad u = a v, grad v = sum a u with a = -sigmoid(-x) resp.
 * sigmoid(x). */
ps_status ps_step_sgns(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg,
                       int64_t B, int32_t window, int32_t n_neg, int64_t out_key_offset,
                       double* loss, void* ws, size_t ws_bytes, void* stream);

/* ps_step_sgns in two phases, as ps_step_kge_prepare / ps_step_kge_apply:
 * the prepare reads only the ids (centre validity, key sort, segments), the
 * apply reads centre, ctx and neg again (the arrays given to the prepare,
 * unchanged, with the same B, window, n_neg and out_key_offset).  Prepare
 * then apply gives exactly the results of ps_step_sgns.  Workspace size:
 * ps_workspace_bytes(num_keys, dim, PS_OP_STEP_SGNS, B, 1 + 2 window
 * (1 + n_neg)).  Staged stores: PS_ERR_UNSUPPORTED. */
ps_status ps_step_sgns_prepare(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                               int32_t window, int32_t n_neg, int64_t out_key_offset, void* ws, size_t ws_bytes,
                               void* stream);
ps_status ps_step_sgns_apply(ps_store* s, const int32_t* centre, const int32_t* ctx, const int32_t* neg, int64_t B,
                             int32_t window, int32_t n_neg, int64_t out_key_offset, double* loss, void* ws,
                             size_t ws_bytes, void* stream);

/* One CTR embedding step (Appendix C, "Click-through-rate prediction",
 * embedding part).  Sample b has F keys keys[b*F + f] and a label in {0,1}:
 *   S = sum_f e_f,  z = sum_{f<g} <e_f, e_g>,  loss = softplus(z) - y z
 *   grad e_f = (sigmoid(z) - y)(S - e_f)
 * keys: device int64[B*F]; label: device float[B]. */
ps_status ps_step_ctr(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F,
                      double* loss, void* ws, size_t ws_bytes, void* stream);

/* ps_step_ctr in two phases, for callers that overlap the key work of the
 * next batch with the table update of this one (two workspaces, two
 * streams), as ps_step_mf_prepare / ps_step_mf_apply do for the MF step.
 * ps_step_ctr_prepare reads only the keys and writes the workspace (sample
 * validity, sort, segments; a sample with a key outside [0, num_keys) is
 * skipped and raises the store's sticky error here); it reads and writes no
 * table row, so it may run while another workspace's apply updates W and G.
 * ps_step_ctr_apply then forms the gradients from the pre-step table, merges
 * them into W and G and writes the loss; it reads the keys again, so keys
 * must be the array given to the prepare, unchanged, and ws the result of
 * that prepare for this store and the same B and F, unmodified.  Ordering
 * prepare before apply (and an apply before the next prepare into the same
 * workspace) is the caller's, e.g. with events.  Prepare then apply gives
 * exactly the results of ps_step_ctr.  Workspace size:
 * ps_workspace_bytes(num_keys, dim, PS_OP_STEP_CTR, B, F).  Staged stores:
 * PS_ERR_UNSUPPORTED. */
ps_status ps_step_ctr_prepare(ps_store* s, const int64_t* keys, int64_t B, int32_t F, void* ws, size_t ws_bytes,
                              void* stream);
ps_status ps_step_ctr_apply(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F,
                            double* loss, void* ws, size_t ws_bytes, void* stream);

/* Synchronize `stream`, then return and clear the store's sticky device
 * error (PS_OK or PS_ERR_KEY_RANGE). */
ps_status ps_get_error(ps_store* s, void* stream);

/* Static description of a status code. */
const char* ps_status_string(ps_status st);

/* Message of the last error raised on the calling thread ("" if none). */
const char* ps_last_error_message(void);

/* Kernel timing (instrumentation).  ps_set_timing(s, mask): bit k of mask
 * turns on timing of kernel id k (PS_TIMING_ALL: every id; 0: off).  The
 * store then brackets each launch of those kernels with HIP events on the
 * launch stream; each event costs a few microseconds of GPU idle time, so a
 * measurement should time only the kernels it reports.  ps_read_timing()
 * synchronizes those events and returns the summed duration (ms) and launch
 * count of one kernel since the last reset, then resets it.  kernel_id: 0 = segmented reduce + AdaGrad, 1 = task gradient
 * (MF: the per-entry record scatter), 2 = radix scatter, 3 = pull, 4 = MF
 * row-key merge that also forms the MF gradients and loss (timed under 4,
 * not 0), 5 = row moves of a staged store between its home tables and its
 * slots (on the staging stream; set the mask while no round runs on the
 * library thread, read it after stopping that thread), 6 = the fp64
 * matrix-core products of the Wide & Deep step, 7 = the unmerged (atomic)
 * update of ps_push_async and ps_step_mf_async. */
#define PS_KERNEL_SEGREDUCE 0
#define PS_KERNEL_TASKGRAD  1
#define PS_KERNEL_SCATTER   2
#define PS_KERNEL_PULL      3
#define PS_KERNEL_MF_ROWMERGE 4
#define PS_KERNEL_STAGE     5
#define PS_KERNEL_MLP       6
#define PS_KERNEL_ASYNC     7
#define PS_TIMING_ALL (-1)
ps_status ps_set_timing(ps_store* s, int32_t mask);
ps_status ps_read_timing(ps_store* s, int32_t kernel_id, double* total_ms, int64_t* launches);

/* Gather probe (instrumentation): reads the rows keys[0..n) of the store's
 * value table the way a gather-bound kernel reads its rows, without that
 * kernel's arithmetic, to measure how fast this part serves a given stream
 * of row reads (the gather ceiling a task kernel is compared with).  keys:
 * device int32[n], read in order by a grid of PS_PROBE_GRID workgroups
 * (row group g of S takes positions g, g + S, ...); keys outside
 * [0, num_keys) are skipped.  sink: device double[PS_PROBE_GRID] receives
 * fp64 partial sums of what was read (their total is the sum of every value
 * read, so the reads cannot be left out).  fp32 stores only (bf16:
 * PS_ERR_UNSUPPORTED); enqueued on `stream`, nothing allocated. */
#define PS_PROBE_GRID 2048
ps_status ps_probe_gather(ps_store* s, const int32_t* keys, int64_t n, double* sink, void* stream);

/* ======================================================================
 * Wide & Deep click-through-rate step (Appendix C, "Click-through-rate
 * prediction": the Wide & Deep model, AdaGrad).
 *
 * Table rows hold [embedding (emb_dim) | wide weight | anything]; only the
 * first emb_dim + 1 values of a row enter the model, the rest get a zero
 * gradient (so AdaGrad leaves them as they are).  For sample b with keys
 * k_f = keys[b*F + f]:
 *   x = concat_f W[k_f][0 .. emb_dim)                    (F*emb_dim values)
 *   h_0 = x;  h_l = relu(h_{l-1} W_l + b_l),  l = 1 .. n_hidden
 *   logit = h_L . w + c + sum_f W[k_f][emb_dim]
 *   loss += softplus(logit) - label[b] * logit
 * The dense parameters are one caller-owned device buffer of fp32 `dense`
 * (and `dense_accum`, their AdaGrad accumulators, same size): for each
 * hidden layer W_l (fan_in x fan_out, row-major, fan_in of the first layer
 * F*emb_dim) then b_l, then w (h_L values) and c (one value).
 * Arithmetic: the MLP forward and backward in fp64 (on the matrix cores);
 * each key occurrence's gradient row [dx_f | dlogit | 0 ...] is rounded to
 * fp32 and merged like every push; the dense gradients are sums over the
 * batch in fp64, rounded once to fp32, then one per-element AdaGrad step
 * with the store's lr and eps.  All gradients come from the pre-step
 * parameters.  A sample with a key outside the table is skipped and
 * flagged (as ps_step_ctr).  hidden: host array of n_hidden (<= 8) widths.
 * The workspace size comes from ps_ctr_wd_workspace_bytes (0 = invalid
 * arguments). */
size_t ps_ctr_wd_workspace_bytes(int64_t num_keys, int32_t dim, int64_t B, int32_t F, int32_t emb_dim,
                                 int32_t n_hidden, const int32_t* hidden);
ps_status ps_step_ctr_wd(ps_store* s, const int64_t* keys, const float* label, int64_t B, int32_t F,
                         int32_t emb_dim, int32_t n_hidden, const int32_t* hidden, float* dense,
                         float* dense_accum, double* loss, void* ws, size_t ws_bytes, void* stream);

/* ======================================================================
 * Staged stores: intent signalling and adaptive action timing
 * (Section 3, "Intent signaling"; Section 4.2, Algorithm 1), for one
 * worker, the GPU, whose full table lives in host memory.
 *
 * The home tables (values and AdaGrad accumulators, num_keys rows each)
 * are caller-owned pinned host memory (hipHostMalloc; torch's
 * pin_memory=True).  HBM holds a table of slots (caller-owned device
 * memory, `values`/`accum` with `row_stride` as in ps_create_strided) and
 * a device map key -> slot (`key_slot`, num_keys int32, caller-owned,
 * filled with -1 by ps_create_staged).  The keys are split into ranges
 * [range_begin[r], range_begin[r+1]) (the last ends at num_keys), each with
 * range_slots[r] slots; a key offset that a step takes (col_key_offset,
 * rel_key_offset, out_key_offset) must begin a range.
 *
 * The worker declares future accesses with ps_intent(keys, C_start,
 * C_end): it will access those keys while its clock C satisfies
 * C_start <= C < C_end (the intent is inactive before, active within,
 * expired after).  ps_advance_clock raises C by one, typically once per
 * batch, before the batch's step.  Rounds (ps_stage_round, or
 * ps_stage_auto's library thread) act on intents: in a round at clock C
 * with Delta = C minus the clock at the previous round, the estimate of
 * clocks per round is smoothed, est <- (1-alpha) est + alpha Delta (not
 * when Delta = 0), and every pending intent with
 * C_start < C + Q_Poiss(2 max(est, Delta), p) is acted upon (Algorithm 1;
 * alpha = 0.1, p = 0.9999, est_0 = 10 unless ps_set_action_timing says
 * otherwise).  Acting makes an intent's keys resident: a key not resident
 * gets a free slot of its range and its home rows are copied in.  A key
 * whose every acted-upon intent has expired is written back to the home
 * tables and its slot freed at the next round.  Intents are acted upon in
 * C_start order; a range with no free slot stops acting until expiries free
 * slots.  An intent still pending when the clock reaches its C_start is
 * acted upon at once inside ps_advance_clock (a forced action, counted).
 *
 * Ordering: the copies of a round run on the store's staging stream after
 * the worker stream's work enqueued before its last ps_advance_clock;
 * ps_advance_clock makes the given worker stream wait for the rounds that
 * staged the intents now active.  So the worker calls ps_advance_clock and
 * the steps on one stream, and every key a step accesses must be covered by
 * an intent that is active at the current clock; an access to a key with no
 * slot is skipped like an invalid id and reported by ps_get_error as
 * PS_ERR_NOT_RESIDENT.  The steps and ps_push take their workspace as for
 * other stores (ps_workspace_bytes covers the id translation) and see the
 * home table's keys; ps_pull reads resident rows.  The two-phase MF step is
 * not available (PS_ERR_UNSUPPORTED).  Home rows of resident keys are stale
 * until ps_stage_flush.  Updates are per-element AdaGrad.
 *
 * ps_create_staged allocates, besides the status block, a staging stream,
 * events, and move lists of 2 x total slots (int64 keys and slots) in
 * device memory and twice that in pinned host memory. */

/* statistics reported by ps_stage_stats, in this order */
#define PS_STAGE_CLOCK      0   /* worker clock */
#define PS_STAGE_ROUNDS     1   /* rounds run */
#define PS_STAGE_FORCED     2   /* forced actions in ps_advance_clock */
#define PS_STAGE_STAGED     3   /* keys copied in, total */
#define PS_STAGE_EVICTED    4   /* keys written back, total */
#define PS_STAGE_RESIDENT   5   /* keys resident now */
#define PS_STAGE_PENDING    6   /* keys of intents not yet acted upon */
#define PS_STAGE_STALLED    7   /* times acting stopped at a full range */
#define PS_STAGE_PLAN_US    8   /* host time of all rounds' planning and enqueueing, microseconds */
#define PS_STAGE_NUM_STATS  9

ps_status ps_create_staged(ps_store** out, int64_t num_keys, int32_t dim, float* home_values,
                           float* home_accum, int64_t home_stride, float* values, float* accum,
                           int64_t row_stride, int32_t* key_slot, int32_t num_ranges,
                           const int64_t* range_begin, const int64_t* range_slots, float lr, float eps,
                           void* stream);

/* Action-timing hyperparameters of Algorithm 1 (0 < alpha <= 1, 0 < p < 1,
 * lambda0 >= 0 resets the estimate). */
ps_status ps_set_action_timing(ps_store* s, double alpha, double p, double lambda0);

/* Intent(keys, c_start, c_end): host array of n keys (duplicates and keys
 * outside [0, num_keys) are allowed and ignored), c_start < c_end.  Cheap:
 * the keys are queued; rounds act on them.  An intent already expired at
 * the current clock is ignored. */
ps_status ps_intent(ps_store* s, const int64_t* keys, int64_t n, int64_t c_start, int64_t c_end);

/* advanceClock: raise the worker clock by one and order `stream` (the
 * worker's) after the staging it now needs, acting at once on intents that
 * became active without a round having acted on them. */
ps_status ps_advance_clock(ps_store* s, void* stream);

/* One round; with wait != 0 the call returns once its copies are done.
 * Not while ps_stage_auto is on. */
ps_status ps_stage_round(ps_store* s, int32_t wait);

/* on != 0: run rounds back to back on a library thread (each lasts until its
 * copies are done); on = 0: stop it and report any error it met. */
ps_status ps_stage_auto(ps_store* s, int32_t on);

/* Write the rows of every resident key back to the home tables (after the
 * work enqueued on `stream`) and wait for it; the keys stay resident. */
ps_status ps_stage_flush(ps_store* s, void* stream);

/* counts[i] for i < n (PS_STAGE_* indices) and the current estimate of
 * clocks per round (either may be NULL when n = 0). */
ps_status ps_stage_stats(ps_store* s, int64_t* counts, int32_t n, double* lambda);

/* The resident keys in ascending order: up to `capacity` into keys (host),
 * their number into *count. */
ps_status ps_stage_resident(ps_store* s, int64_t* keys, int64_t capacity, int64_t* count);

/* Algorithm 1 as a pure host function: from the previous estimate, the
 * clock at the previous round and now, return the new estimate and the
 * horizon H (act on an intent iff C_start < H). */
ps_status ps_action_timing(double lambda_prev, int64_t c_prev, int64_t c_now, double alpha, double p,
                           double* lambda_new, int64_t* horizon);

#ifdef __cplusplus
}
#endif
#endif /* ADAPM_H */
