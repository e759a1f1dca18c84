/*
 * tc.h - tensor-group collectives and the fused elastic-averaging SGD step
 * for AMD Instinct MI355X (gfx950).
 *
 * The method is that of MXNET-MPI (Mamidala, Kollias, Ward, Artico, arXiv
 * 1801.03855): a worker's per-layer tensors are handled as one object, K
 * per-worker copies of it are summed or averaged, and the averaging is fused
 * with the elastic-averaging SGD update.  Here the K workers' copies are K
 * buffers resident in one GPU's memory.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Plain C ABI.  Pointers marked "device" point to GPU memory of the device
 *   that was current when the group was created; arrays of such pointers
 *   (x[], grad[], in[], flat[], tensors[]) are HOST arrays that the call
 *   reads before it returns.
 * - All data buffers are owned by the caller.  The library owns only the
 *   descriptors it returns (tc_group, tc_tensorlist) and their device tables.
 * - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *   Every data operation is enqueued asynchronously on it, and nothing waits
 *   for it to finish; faults during execution surface at the caller's next
 *   synchronisation.
 * - Data operations allocate nothing, copy nothing between host and device
 *   and never synchronise: they only enqueue kernels, whose arguments carry
 *   the pointers of the call.  A sequence of them can be captured in a HIP
 *   graph and replayed; the descriptors it names (and their device tables)
 *   must then outlive the graph.  Only tc_group_create/_destroy and
 *   tc_tensorlist_create/_destroy allocate, copy and free.
 * - Return value of the data operations: TC_OK, or a negative tc_status.
 *   On error nothing has been enqueued, except TC_EHIP from a failed launch;
 *   tc_last_error() then describes the error (thread-local, valid until the
 *   next call on the same thread).
 * - A flat buffer of a group holds N = sum(sizes) elements, densely
 *   concatenated in tensor order with no padding.  Buffers need only the
 *   alignment of their element type; 16-byte aligned buffers take the
 *   vectorised path.
 * - Binary32 arithmetic, round to nearest even, no flush of subnormals.
 *   bfloat16 inputs are widened exactly to binary32.
 */
#ifndef TC_H
#define TC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tc_group tc_group;           /* opaque, library-owned */
typedef struct tc_tensorlist tc_tensorlist; /* opaque, library-owned */

typedef enum { TC_SUM = 0, TC_AVG = 1 } tc_op;
typedef enum { TC_F32 = 0, TC_BF16 = 1 } tc_dtype;
typedef enum {
    TC_OK = 0,
    TC_EINVAL = -1,       /* bad argument; nothing enqueued */
    TC_ENOMEM = -2,       /* a device or host allocation failed */
    TC_EHIP = -3,         /* a HIP call or kernel launch failed */
    TC_EUNSUPPORTED = -4  /* valid request the library does not implement */
} tc_status;

/* Largest number of worker copies K accepted by any entry point. */
#define TC_MAX_K 64

/* Thread-local description of the last error on this thread ("" if none). */
const char* tc_last_error(void);

/* Library version, major*10000 + minor*100 + patch. */
int32_t tc_version(void);

/* ------------------------------------------------------------------------
 * Tensor group descriptor.
 *
 * A group is the ordered list of a model's layer tensors (one key per weight
 * tensor, Sec. 3.2 of the paper; the keys visited in tensor order, Sec. 5)
 * treated as one flat object (the "tensor" of Sec. 6.1).  Tensor t occupies
 * flat positions [offsets[t], offsets[t+1]), offsets[0] = 0, offsets[t+1] =
 * offsets[t] + sizes[t].
 *
 * tc_group_create: sizes is a host array of n >= 1 element counts, each
 * >= 0 (zero-size tensors are allowed); it is copied.  Builds the offset
 * table and, for each way the kernels cut the group into chunks (separate
 * buffers, tensor-layout pack/unpack, the pipelined step), a table of each
 * chunk's first tensor, and copies them to the current device
 * (synchronously; this is set-up, not part of a step).  Returns NULL on
 * error (n < 1, a negative size, a total that overflows int64, allocation
 * failure, no device); see tc_last_error.
 * ---------------------------------------------------------------------- */
tc_group* tc_group_create(const int64_t* sizes, int32_t n);

/* Frees the group and its device tables.  NULL-safe.  Must not be called
 * while work that uses the group is still pending on a stream. */
void tc_group_destroy(tc_group* g);

/* N = sum of the sizes, or -1 if g is NULL. */
int64_t tc_group_numel(const tc_group* g);

/* Number of tensors n, or -1 if g is NULL. */
int32_t tc_group_ntensors(const tc_group* g);

/* Copies the n+1 offsets into the host array out.  TC_EINVAL on NULL. */
int32_t tc_group_offsets(const tc_group* g, int64_t* out);

/* ------------------------------------------------------------------------
 * Tensor list: K copies of a group held as separate per-layer tensors (the
 * paper's "tensorlist", Sec. 3.2: for every key one tensor per worker).
 *
 * ptrs is a host array of K*n device pointers, copy-major: ptrs[k*n + t] is
 * tensor t of copy k and holds sizes[t] elements of `dtype`, contiguous,
 * aligned to the element size.  A zero-size tensor's pointer may be NULL.
 * The pointer table is copied to the device once (synchronously); the
 * tensors themselves stay owned by the caller and must outlive the list.
 * Returns NULL on error (K outside [1, TC_MAX_K], a NULL pointer for a
 * non-empty tensor, misalignment, bad dtype, allocation failure).
 * ---------------------------------------------------------------------- */
tc_tensorlist* tc_tensorlist_create(const tc_group* g, int32_t K,
                                    const void* const* ptrs, int32_t dtype);

/* Frees the list's device table.  NULL-safe.  The group must outlive it. */
void tc_tensorlist_destroy(tc_tensorlist* tl);

/* ------------------------------------------------------------------------
 * tc_pack: gather every copy's tensors into its flat buffer,
 *   flat[k][offsets[t] + e] = tensor(k, t)[e]      for all k < K, t, e,
 * bit for bit (push collects the key list, Sec. 3.2).  flat is a host array
 * of K device pointers, each to N elements of the list's dtype.  One launch
 * for all K copies and all n tensors.  Flat buffers must not overlap the
 * tensors or each other.
 * ---------------------------------------------------------------------- */
int32_t tc_pack(const tc_tensorlist* tl, void* const* flat, void* stream);

/* ------------------------------------------------------------------------
 * tc_unpack: scatter every copy's flat buffer back to its tensors,
 *   tensor(k, t)[e] = flat[k][offsets[t] + e],
 * bit for bit (pull copies the value to every tensor of the list,
 * Sec. 3.2).  Same layout and rules as tc_pack.
 * ---------------------------------------------------------------------- */
int32_t tc_unpack(const tc_tensorlist* tl, const void* const* flat, void* stream);

/* ------------------------------------------------------------------------
 * tc_reduce: K-way reduction of flat copies (the tensor reduction of
 * Sec. 6.3 and Sec. 7.3; push sums the tensors of a key, Sec. 3.2; the
 * synchronous SGD rescale by 1/mini_batch_size makes it an average, Sec. 5):
 *   out[j] = in_0[j] + ... + in_{K-1}[j]          (TC_SUM)
 *   out[j] = (in_0[j] + ... + in_{K-1}[j]) / K    (TC_AVG)
 * for j < N.  in is a host array of K device pointers to N binary32 values;
 * out is a device pointer to N binary32 values.  The K terms are added as a
 * pairwise tree (adjacent pairs, level by level; an odd last term is carried
 * up), and AVG divides the sum by K with one correctly rounded division; so
 * the AVG of K identical copies returns the copy exactly for power-of-two K.
 * out may be identical to one of the inputs (in place); a partial overlap
 * returns TC_EINVAL.  K in [1, TC_MAX_K].
 * ---------------------------------------------------------------------- */
int32_t tc_reduce(const tc_group* g, int32_t K, const float* const* in,
                  float* out, int32_t op, void* stream);

/* As tc_reduce, with inputs of type in_dtype (TC_F32 or TC_BF16); the sum
 * is accumulated and returned in binary32.  In place is allowed for TC_F32
 * inputs only: a binary32 output element is twice as wide as a bfloat16
 * input element, so an output written over a bfloat16 input would overwrite
 * input elements that other lanes have not yet read.  With TC_BF16 inputs,
 * an out that overlaps any input returns TC_EINVAL. */
int32_t tc_reduce_ex(const tc_group* g, int32_t K, const void* const* in,
                     int32_t in_dtype, float* out, int32_t op, void* stream);

/* ------------------------------------------------------------------------
 * easgd_step: one synchronous elastic-averaging SGD step over K workers,
 * fused with the K-way reduction of the center's elastic term, in place.
 * For every j < N, with c = x_c[j] and x_i = x[i][j] read before any write:
 *
 *   d_i       = x_i - c
 *   x[i][j]   = x_i - eta * (grad_i[j] + rho * d_i)
 *   x_c[j]    = c + (eta*rho) * (d_0 + ... + d_{K-1})
 *
 * The worker line is the client's elastic move (Sec. 2.2, Eq. 3, with
 * alpha = eta*rho) followed by the SGD move -eta*g (Sec. 2.1, Eq. 1); the
 * center line is the server's elastic move (Sec. 2.2, Eq. 2) summed over
 * the K workers.  Arithmetic: d_i = x_i - c; t = fma(rho, d_i, g_i);
 * x_i' = fma(-eta, t, x_i); the d_i are summed by the same pairwise tree as
 * tc_reduce; x_c' = fma(eta*rho, sum, c), with eta*rho rounded once to
 * binary32.
 *
 * x: host array of K device pointers to N binary32 worker values (in/out),
 * pairwise distinct.  grad: host array of K device pointers to N binary32
 * gradients (read only; may alias each other, not x or x_c).  x_c: device
 * pointer to N binary32 center values (in/out), distinct from all others.
 * eta, rho: finite.  TC_EINVAL on K outside [1, TC_MAX_K], NULL pointers
 * with N > 0, non-finite eta or rho.
 * ---------------------------------------------------------------------- */
int32_t easgd_step(const tc_group* g, int32_t K, float* const* x,
                   const float* const* grad, float* x_c, float eta, float rho,
                   void* stream);

/* As easgd_step, with gradients of type g_dtype (TC_F32 or TC_BF16). */
int32_t easgd_step_ex(const tc_group* g, int32_t K, float* const* x,
                      const void* const* grad, int32_t g_dtype, float* x_c,
                      float eta, float rho, void* stream);

/* ------------------------------------------------------------------------
 * reduce_easgd_step: the K-way reduction of the gradients (the push's sum
 * over the tensors of a key, Sec. 3.2, and its average as SGD.Update's
 * rescale gives it, Sec. 5) fused with the elastic step above (Sec. 2.2,
 * Eqs. 2 and 3, summed over K workers, with the SGD move of Sec. 2.1), in
 * one pass that reads each gradient once.  Equivalent, bit for bit, to
 *     tc_reduce_ex(g, K, grad, g_dtype, out, op);
 *     easgd_step_ex(g, K, x, grad, g_dtype, x_c, eta, rho);
 * (the sums use the same pairwise tree, AVG the same single rounding of
 * SUM / K).  Arguments as easgd_step_ex, plus out: device pointer to N
 * binary32 values (written), overlapping none of x, grad, x_c; op: TC_SUM
 * or TC_AVG.  TC_EINVAL on bad arguments, NULL out with N > 0 included.
 * ---------------------------------------------------------------------- */
int32_t reduce_easgd_step(const tc_group* g, int32_t K, float* const* x,
                          const void* const* grad, int32_t g_dtype, float* x_c,
                          float* out, int32_t op, float eta, float rho, void* stream);

/* ------------------------------------------------------------------------
 * Tensor layout.  The paper's "tensor" (Sec. 6.1) collects one vector per
 * worker and treats the set as a single unit.  In this layout the K
 * copies of a group live in ONE buffer, interleaved in slots of four
 * consecutive elements: element e of copy i is at index
 *
 *     ((e / 4) * K + i) * 4 + (e % 4),
 *
 * so slot j holds, one after the other, the j-th four elements of copy 0,
 * copy 1, ..., copy K-1.  The buffer holds tc_tensor_numel(g, K) =
 * ceil(N/4) * 4 * K elements; when N is not a multiple of 4 the positions of
 * e >= N in the last slot are padding, never read or written.  A K-way
 * operation then reads one stream instead of K (on MI355X the fused step
 * runs ~15% faster than on K separate buffers).  Results are the same as the
 * separate-buffer entry points': the K-way sums use the same pairwise tree
 * (bit-identical for power-of-two K, identical up to the sign of a zero
 * otherwise).  Every buffer passed to these calls must be 16-byte aligned
 * (TC_EINVAL otherwise).
 * ---------------------------------------------------------------------- */

/* Elements of a K-copy tensor-layout buffer of group g, or -1 on bad
 * arguments. */
int64_t tc_tensor_numel(const tc_group* g, int32_t K);

/* Pack the K copies' separate tensors (the list's K*n tensors) into one
 * tensor-layout buffer of the list's dtype (Sec. 3.2 push + Sec. 6.1
 * tensor): tensor[((e/4)*K + k)*4 + e%4] = tensor(k, t)[e - offsets[t]] for
 * the tensor t holding flat element e.  Bit for bit; one launch. */
int32_t tc_pack_tensor(const tc_tensorlist* tl, void* tensor, void* stream);

/* The inverse scatter (Sec. 3.2 pull): every copy's separate tensors from
 * one tensor-layout buffer. */
int32_t tc_unpack_tensor(const tc_tensorlist* tl, const void* tensor, void* stream);

/* tc_reduce_ex on a tensor-layout input: out[e] = sum over i of copy i's
 * element e (or that / K), for e < N.  in: K copies of in_dtype in the
 * tensor layout; out: N binary32 values, not overlapping in. */
int32_t tc_reduce_tensor(const tc_group* g, int32_t K, const void* in, int32_t in_dtype,
                         float* out, int32_t op, void* stream);

/* easgd_step_ex on tensor-layout workers and gradients: the same update,
 * in place on x (K binary32 copies in the tensor layout) and x_c (N binary32
 * values), with grad (K copies of g_dtype in the tensor layout).  The three
 * buffers must not overlap. */
int32_t easgd_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad,
                          int32_t g_dtype, float* x_c, float eta, float rho, void* stream);

/* reduce_easgd_step on tensor-layout workers and gradients: bit for bit
 * tc_reduce_tensor(g, K, grad, g_dtype, out, op) followed by
 * easgd_step_tensor(g, K, x, grad, g_dtype, x_c, eta, rho).  out: N binary32
 * values, 16-byte aligned, overlapping none of x, grad, x_c. */
int32_t reduce_easgd_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad,
                                 int32_t g_dtype, float* x_c, float* out, int32_t op,
                                 float eta, float rho, void* stream);

/* ------------------------------------------------------------------------
 * The ESGD schedule with a communication period (Sec. 5, the ESGD listing:
 * SGD.Update every iteration, the elastic exchange every INTERVAL = 64
 * iterations) and its pieces.
 *
 * sgd_step: plain SGD on every worker, in place (Sec. 2.1, Eq. 1, dw =
 * -eta g; SGD.Update's rescale folded into eta):
 *     x[i][j] = fma(-eta, grad[i][j], x[i][j]).
 * x: K device pointers to N binary32 values, pairwise disjoint; grad: K
 * device pointers to N values of g_dtype, not overlapping any x.
 * ---------------------------------------------------------------------- */
int32_t sgd_step(const tc_group* g, int32_t K, float* const* x, const void* const* grad,
                 int32_t g_dtype, float eta, void* stream);

/* sgd_step on tensor-layout workers and gradients (16-byte aligned,
 * disjoint). */
int32_t sgd_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad,
                        int32_t g_dtype, float eta, void* stream);

/* One iteration of the periodic schedule: easgd_step_ex when
 * iteration % tau == 0, else sgd_step (x_c untouched).  tau >= 1,
 * iteration >= 0; arguments as for those two calls. */
int32_t easgd_period_step(const tc_group* g, int32_t K, float* const* x,
                          const void* const* grad, int32_t g_dtype, float* x_c, float eta,
                          float rho, int64_t iteration, int32_t tau, void* stream);

/* The same on the tensor layout (easgd_step_tensor / sgd_step_tensor). */
int32_t easgd_period_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad,
                                 int32_t g_dtype, float* x_c, float eta, float rho,
                                 int64_t iteration, int32_t tau, void* stream);

/* ------------------------------------------------------------------------
 * elastic_async: asynchronous elastic averaging, one worker at a time
 * (Sec. 2.2, Eqs. 2 and 3; Sec. 5, the asynchronous ESGD listing: a
 * worker's push makes the server apply Elastic1 to the center and the
 * worker applies Elastic2).  For r = 0 .. R-1 in turn, with w = order[r]
 * and d = x_w - c from the values before this exchange:
 *     c   = fma(alpha, d, c)          (the center moves toward the worker)
 *     x_w = fma(-alpha, d, x_w)       (the worker moves toward the center)
 * so later exchanges see the center left by earlier ones; each exchange
 * leaves x_w + c unchanged in exact arithmetic.  order: host array of R
 * worker indices in [0, K), no worker twice (0 <= R <= K; R = 0 is a
 * no-op); alpha finite.  x: K disjoint binary32 buffers; x_c: N binary32
 * values not overlapping them.
 * ---------------------------------------------------------------------- */
int32_t elastic_async(const tc_group* g, int32_t K, float* const* x, float* x_c,
                      const int32_t* order, int32_t R, float alpha, void* stream);

/* elastic_async on tensor-layout workers (16-byte aligned x and x_c). */
int32_t elastic_async_tensor(const tc_group* g, int32_t K, float* x, float* x_c,
                             const int32_t* order, int32_t R, float alpha, void* stream);

/* ------------------------------------------------------------------------
 * sync_sgd_step: synchronous SGD through pushpull (Sec. 5, the synchronous
 * SGD listing; Sec. 4.2, pushpull): with S = the pairwise sum of the K
 * gradients (the value push and pull leave in every worker's gradient),
 *     x[i][j] = fma(-(eta*rescale), S[j], x[i][j])   for every worker i,
 * eta*rescale rounded once to binary32 (rescale = 1/mini_batch_size
 * averages).  With broadcast != 0, every grad[i] is overwritten with S (the
 * pull's copy to every tensor); binary32 gradients only (TC_EUNSUPPORTED
 * for bfloat16).  x: K disjoint binary32 buffers; grad: K buffers of
 * g_dtype not overlapping x (and pairwise disjoint when broadcast).
 * ---------------------------------------------------------------------- */
int32_t sync_sgd_step(const tc_group* g, int32_t K, float* const* x, void* const* grad,
                      int32_t g_dtype, float eta, float rescale, int32_t broadcast, void* stream);

/* sync_sgd_step on tensor-layout workers and gradients. */
int32_t sync_sgd_step_tensor(const tc_group* g, int32_t K, float* x, void* grad,
                             int32_t g_dtype, float eta, float rescale, int32_t broadcast,
                             void* stream);

/* ------------------------------------------------------------------------
 * tc_broadcast: dst[i][j] = src[j] for every copy i < K, bit for bit (the
 * pull copies the value to every tensor of the list, Sec. 3.2; the tensor
 * broadcast of Sec. 6.3.1).  src: N elements of dtype; dst: K disjoint
 * buffers of N elements, not overlapping src.
 * ---------------------------------------------------------------------- */
int32_t tc_broadcast(const tc_group* g, int32_t K, const void* src, void* const* dst,
                     int32_t dtype, void* stream);

/* tc_broadcast into every copy of one tensor-layout buffer (16-byte
 * aligned src and dst). */
int32_t tc_broadcast_tensor(const tc_group* g, int32_t K, const void* src, void* dst,
                            int32_t dtype, void* stream);

/* ------------------------------------------------------------------------
 * easgd_pipeline_tensor: the whole step in one pass over the tensor layout.
 * Equivalent, bit for bit, to the four calls
 *     tc_pack_tensor(grads, g_tensor);
 *     tc_reduce_tensor(g, K, g_tensor, grads' dtype, gbar, TC_AVG);
 *     easgd_step_tensor(g, K, x, g_tensor, grads' dtype, x_c, eta, rho);
 *     tc_unpack_tensor(params, x);
 * but each workgroup takes its chunk of the group through all four with the
 * intermediates on chip, so the gradients are read once and the new workers
 * are not read back: the on-chip form of pipelining the pieces of a chunked
 * reduction through its stages (Sec. 6.3.2, the multi-ring listing), for
 * the push (Sec. 3.2: gather and sum a key's tensors), the elastic update
 * (Sec. 2.2, Eqs. 2 and 3, summed over K workers, with the SGD move of
 * Sec. 2.1) and the pull (Sec. 3.2: copy to every tensor of the list).
 *
 * grads: K*n gradient tensors (TC_F32 or TC_BF16); params: K*n binary32
 * tensors; both lists of the same group object and K.  g_tensor: the packed
 * gradients in the tensor layout (tc_tensor_numel(g, K) elements of the
 * gradient dtype), or NULL to leave them unwritten.  gbar: N binary32
 * values (the AVG).  x: the K binary32 workers in the tensor layout (in/out).
 * x_c: N binary32 values (in/out).  Every flat buffer 16-byte aligned and
 * disjoint from the others; the per-layer tensors must not overlap any flat
 * buffer or each other (not checked).  eta, rho finite.  TC_EINVAL on bad
 * arguments.
 * ---------------------------------------------------------------------- */
int32_t easgd_pipeline_tensor(const tc_tensorlist* grads, const tc_tensorlist* params, void* g_tensor,
                              float* gbar, float* x, float* x_c, float eta, float rho, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TC_H */
