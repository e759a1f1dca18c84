/*
 * CPU oracle for the tensor-group collective reduction and the synchronous
 * elastic-averaging SGD step of MXNET-MPI (Mamidala, Kollias, Ward, Artico,
 * "MXNET-MPI: Embedding MPI parallelism in Parameter Server Task Model for
 * scaling Deep Learning", arXiv 1801.03855).
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark load this library.  The product path never
 * links, loads or calls it, and it shares no source, header, table or helper
 * with the GPU library.
 *
 * Precision: every floating-point result is computed in IEEE binary64 from
 * the exact values of the stored inputs (binary32, or bfloat16 decoded from
 * its bit fields) and returned in binary64.  The code is deliberately plain:
 * one element at a time, in the order the definitions are written, with no
 * blocking, vectorisation or reordering.
 *
 * Passages followed (sections and equations of the paper):
 *   group offsets   Sec. 3.2: one key per weight tensor of the model; Sec. 5:
 *                   the training loop visits the keys in tensor order;
 *                   Sec. 6.1: a set of vectors treated as a single unit.
 *   pack / unpack   Sec. 3.2: push gathers the tensors of the key list, pull
 *                   copies a value back to every tensor of the list.
 *   reduce          Sec. 2.2: workers wait for the global average of the
 *                   locally computed gradients; Sec. 3.2: push first sums
 *                   the tensors of one key; Sec. 5 (synchronous SGD): the
 *                   sum is rescaled by 1/mini_batch_size, i.e. averaged.
 *   sgd step        Sec. 2.1, Eq. (1) with dw = -eta * g; Sec. 5 listings:
 *                   SGD.Update(params, grads, rescale) scales the step by
 *                   rescale, folded here into eta.
 *   async exchange  Sec. 2.2, Eqs. (2) and (3) for one worker at a time:
 *                   the asynchronous elastic averaging of the ESGD listing
 *                   (Sec. 5), where each worker's push updates the center
 *                   (Elastic1) and the worker moves toward the center
 *                   (Elastic2), workers in arrival order.
 *   sync pushpull   Sec. 5, synchronous SGD: push and pull (or pushpull,
 *                   Sec. 4.2) leave every worker's gradient equal to the sum
 *                   over the workers; SGD.Update then applies it with rescale
 *                   1/mini_batch_size.
 *   broadcast       Sec. 3.2: pull copies one value to every tensor of the
 *                   list.
 *   tensor layout   Sec. 6.1: a "tensor" collects one vector per worker and
 *                   treats the set as a single unit.  Here the K copies
 *                   are held in one buffer, interleaved in slots of four
 *                   consecutive elements (an index map of this library's
 *                   design, written out plainly below).
 *   easgd step      Sec. 2.1, Eq. (1) with dw = -eta * g (plain SGD);
 *                   Sec. 2.2, Eqs. (2) and (3) (elastic averaging: center
 *                   moves toward the worker, worker moves toward the center,
 *                   both by alpha times their difference), taken over K
 *                   workers at once with alpha = eta * rho, every update
 *                   reading the time-t values.
 */

#include <math.h>
#include <stdint.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1
#define ORACLE_SUM 0
#define ORACLE_AVG 1

/*
 * Value of one bfloat16 code, from the format's fields: 1 sign bit, 8
 * exponent bits (bias 127), 7 fraction bits.  Exponent 0 encodes zero and
 * subnormals (fraction/128 * 2^-126), exponent 255 encodes infinities and
 * NaNs, anything else (1 + fraction/128) * 2^(exponent - 127).
 */
static double bf16_value(uint16_t code)
{
    int sign = (code >> 15) & 1;
    int expo = (code >> 7) & 0xFF;
    int frac = code & 0x7F;
    double mag;
    if (expo == 0)
        mag = ldexp((double)frac / 128.0, -126);
    else if (expo == 255)
        mag = frac ? NAN : INFINITY;
    else
        mag = ldexp(1.0 + (double)frac / 128.0, expo - 127);
    return sign ? -mag : mag;
}

/* Exact value of element j of a stored array of the given type. */
static double stored_value(const void* base, int32_t dtype, int64_t j)
{
    if (dtype == ORACLE_BF16)
        return bf16_value(((const uint16_t*)base)[j]);
    return (double)((const float*)base)[j];
}

/* Decode n stored elements to their exact binary64 values. */
void oracle_widen(const void* in, int32_t dtype, int64_t n, double* out)
{
    for (int64_t j = 0; j < n; ++j)
        out[j] = stored_value(in, dtype, j);
}

/*
 * Group offsets: tensor t of the group occupies flat positions
 * [offsets[t], offsets[t+1]); offsets[0] = 0 and each tensor starts where
 * the previous one ends (dense concatenation in key order).  Returns the
 * flat length N = offsets[n].
 */
int64_t oracle_group_offsets(const int64_t* sizes, int32_t n, int64_t* offsets)
{
    offsets[0] = 0;
    for (int32_t t = 0; t < n; ++t)
        offsets[t + 1] = offsets[t] + sizes[t];
    return offsets[n];
}

/*
 * Pack: flat[offsets[t] + e] = tensor_t[e] for every tensor t and element e,
 * copied bit for bit (elem_bytes = 4 for binary32, 2 for bfloat16).
 */
void oracle_pack(int32_t n, const int64_t* sizes, const void* const* tensors,
                 int32_t elem_bytes, void* flat)
{
    unsigned char* dst = (unsigned char*)flat;
    int64_t start = 0;
    for (int32_t t = 0; t < n; ++t) {
        const unsigned char* src = (const unsigned char*)tensors[t];
        for (int64_t e = 0; e < sizes[t]; ++e)
            memcpy(dst + (start + e) * elem_bytes, src + e * elem_bytes,
                   (size_t)elem_bytes);
        start += sizes[t];
    }
}

/* Unpack: tensor_t[e] = flat[offsets[t] + e], bit for bit. */
void oracle_unpack(int32_t n, const int64_t* sizes, const void* flat,
                   int32_t elem_bytes, void* const* tensors)
{
    const unsigned char* src = (const unsigned char*)flat;
    int64_t start = 0;
    for (int32_t t = 0; t < n; ++t) {
        unsigned char* dst = (unsigned char*)tensors[t];
        for (int64_t e = 0; e < sizes[t]; ++e)
            memcpy(dst + e * elem_bytes, src + (start + e) * elem_bytes,
                   (size_t)elem_bytes);
        start += sizes[t];
    }
}

/*
 * Reduce K flat copies: out[j] = in_0[j] + ... + in_{K-1}[j] (SUM), or that
 * sum divided by K (AVG).
 */
void oracle_reduce(int32_t K, int64_t N, const void* const* in, int32_t dtype,
                   int32_t op, double* out)
{
    for (int64_t j = 0; j < N; ++j) {
        double sum = 0.0;
        for (int32_t i = 0; i < K; ++i)
            sum += stored_value(in[i], dtype, j);
        out[j] = (op == ORACLE_AVG) ? sum / (double)K : sum;
    }
}

/*
 * One synchronous elastic-averaging SGD step over K workers, in place.
 * For every element j, with c = xc[j] and x_i = x[i][j] at time t:
 *
 *   center:  xc[j]   = c + eta*rho * sum_i (x_i - c)
 *   worker:  x[i][j] = x_i - eta * (g_i + rho * (x_i - c))
 *
 * The worker line is the elastic move x_i - alpha*(x_i - c) followed by the
 * SGD move -eta*g_i, with alpha = eta*rho; the center line is the center's
 * elastic move summed over the K workers.  Both read time-t values only.
 * x and xc hold binary64 state; g holds the stored gradients.
 */
void oracle_easgd_step(int32_t K, int64_t N, double* const* x,
                       const void* const* g, int32_t g_dtype, double* xc,
                       double eta, double rho)
{
    double alpha = eta * rho;
    for (int64_t j = 0; j < N; ++j) {
        double c = xc[j];
        double spread = 0.0;
        for (int32_t i = 0; i < K; ++i)
            spread += x[i][j] - c;
        for (int32_t i = 0; i < K; ++i) {
            double xi = x[i][j];
            double gi = stored_value(g[i], g_dtype, j);
            x[i][j] = xi - eta * (gi + rho * (xi - c));
        }
        xc[j] = c + alpha * spread;
    }
}

/*
 * Tensor layout of K copies of a group of N elements: element e of copy i
 * sits at index ((e / 4) * K + i) * 4 + (e % 4) of one buffer of
 * ceil(N / 4) * 4 * K elements.  Positions for e >= N are padding and are
 * left untouched.
 */
static int64_t tensor_index(int32_t K, int64_t e, int32_t i)
{
    return ((e / 4) * K + i) * 4 + (e % 4);
}

/* Gather K flat copies into the tensor layout, bit for bit. */
void oracle_tensor_from_copies(int32_t K, int64_t N, const void* const* copies,
                               int32_t elem_bytes, void* tensor)
{
    unsigned char* dst = (unsigned char*)tensor;
    for (int32_t i = 0; i < K; ++i)
        for (int64_t e = 0; e < N; ++e)
            memcpy(dst + tensor_index(K, e, i) * elem_bytes,
                   (const unsigned char*)copies[i] + e * elem_bytes,
                   (size_t)elem_bytes);
}

/* Scatter the tensor layout back into K flat copies, bit for bit. */
void oracle_copies_from_tensor(int32_t K, int64_t N, const void* tensor,
                               int32_t elem_bytes, void* const* copies)
{
    const unsigned char* src = (const unsigned char*)tensor;
    for (int32_t i = 0; i < K; ++i)
        for (int64_t e = 0; e < N; ++e)
            memcpy((unsigned char*)copies[i] + e * elem_bytes,
                   src + tensor_index(K, e, i) * elem_bytes,
                   (size_t)elem_bytes);
}

/*
 * Plain SGD on K workers, in place: x[i][j] = x_i - eta * g_i.
 */
void oracle_sgd_step(int32_t K, int64_t N, double* const* x, const void* const* g,
                     int32_t g_dtype, double eta)
{
    for (int32_t i = 0; i < K; ++i)
        for (int64_t j = 0; j < N; ++j)
            x[i][j] = x[i][j] - eta * stored_value(g[i], g_dtype, j);
}

/*
 * Asynchronous elastic exchanges, in place: for each worker w = order[r],
 * r = 0 .. R-1 in turn, with d = x_w - c taken from the values before this
 * exchange,
 *   center:  c   = c + alpha * d      (Elastic1, on the server)
 *   worker:  x_w = x_w - alpha * d    (Elastic2, on the client)
 * so each later exchange sees the center left by the earlier ones.
 */
void oracle_elastic_async(int32_t K, int64_t N, double* const* x, double* xc,
                          const int32_t* order, int32_t R, double alpha)
{
    (void)K;
    for (int64_t j = 0; j < N; ++j)
        for (int32_t r = 0; r < R; ++r) {
            int32_t w = order[r];
            double d = x[w][j] - xc[j];
            xc[j] = xc[j] + alpha * d;
            x[w][j] = x[w][j] - alpha * d;
        }
}

/*
 * Synchronous SGD through pushpull: with S_j = g_0[j] + ... + g_{K-1}[j]
 * (the value push/pull leave in every worker's gradient),
 *   x[i][j] = x_i - eta * rescale * S_j    for every worker i,
 * and, when broadcast is set, every g_i[j] becomes S_j (returned in the
 * binary64 array sum_out, which the caller compares with each copy).
 */
void oracle_sync_sgd(int32_t K, int64_t N, double* const* x, const void* const* g,
                     int32_t g_dtype, double eta, double rescale, double* sum_out)
{
    for (int64_t j = 0; j < N; ++j) {
        double S = 0.0;
        for (int32_t i = 0; i < K; ++i)
            S += stored_value(g[i], g_dtype, j);
        for (int32_t i = 0; i < K; ++i)
            x[i][j] = x[i][j] - eta * rescale * S;
        if (sum_out)
            sum_out[j] = S;
    }
}

/* Broadcast: dst_i[j] = src[j] for every copy i, bit for bit. */
void oracle_broadcast(int32_t K, int64_t N, const void* src, int32_t elem_bytes,
                      void* const* dst)
{
    for (int32_t i = 0; i < K; ++i)
        memcpy(dst[i], src, (size_t)(N * elem_bytes));
}
