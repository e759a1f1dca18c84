// C entry points: argument validation, descriptors, dispatch to launchers.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "tc_internal.h"

namespace tc {

static thread_local std::string t_error;

void set_error(const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_error = buf;
}

void clear_error() { t_error.clear(); }

namespace {

int32_t fail(int32_t code, const char* what) {
    set_error("%s", what);
    return code;
}

int32_t hip_fail(hipError_t e, const char* where) {
    set_error("%s: %s", where, hipGetErrorString(e));
    return TC_EHIP;
}

int elem_size(int32_t dtype) { return dtype == TC_BF16 ? 2 : dtype == TC_F32 ? 4 : 0; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// [p, p + bytes) and [q, q + bytes2) share a byte.
bool overlap(const void* p, int64_t bytes, const void* q, int64_t bytes2) {
    auto a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
    return a < b + static_cast<uintptr_t>(bytes2) && b < a + static_cast<uintptr_t>(bytes);
}

// The group's device must be the current one.
int32_t check_device(const tc_group* g) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != g->device) {
        set_error("the group lives on device %d but device %d is current", g->device, dev);
        return TC_EINVAL;
    }
    return TC_OK;
}

}  // namespace
}  // namespace tc

using namespace tc;

TC_API const char* tc_last_error(void) { return t_error.c_str(); }

TC_API int32_t tc_version(void) { return 100; }

// ---------------------------------------------------------------- groups

TC_API tc_group* tc_group_create(const int64_t* sizes, int32_t n) {
    clear_error();
    if (n < 1) { set_error("n must be >= 1 (got %d)", n); return nullptr; }
    if (!sizes) { set_error("sizes is NULL"); return nullptr; }
    auto* g = new (std::nothrow) tc_group();
    if (!g) { set_error("out of host memory"); return nullptr; }
    g->n = n;
    g->sizes.assign(sizes, sizes + n);
    g->offsets.resize(static_cast<size_t>(n) + 1);
    g->offsets[0] = 0;
    for (int32_t t = 0; t < n; ++t) {
        if (sizes[t] < 0) { set_error("sizes[%d] = %lld is negative", t, (long long)sizes[t]); delete g; return nullptr; }
        if (sizes[t] > INT64_MAX / 8 - g->offsets[t]) { set_error("group too large"); delete g; return nullptr; }
        g->offsets[t + 1] = g->offsets[t] + sizes[t];
    }
    g->N = g->offsets[n];
    g->large = g->N / n >= TC_PACK_LARGE_MEAN;
    g->sep.chunk = g->large ? TC_PACK_CHUNK_LARGE : TC_PACK_CHUNK_SMALL;
    g->tpack.chunk = TC_TPACK_CHUNK;
    g->tpack_fine.chunk = TC_TPACK_CHUNK_FINE;
    g->pipe.chunk = TC_PIPE_CHUNK;
    g->pipe_fine.chunk = TC_PIPE_CHUNK_FINE;
    // 2-byte elements on groups of large tensors: chunks of twice the
    // elements, the bytes of a binary32 chunk (measured on MI355X, bfloat16
    // pack and unpack on ResNet-50 at K = 2-16 and VGG-16 at K = 4: 13-17%
    // faster than 2,048 elements; on 10,000 small tensors 8,192 elements
    // against 4,096 measured +12% to -5%, and they keep 4,096)
    g->sep2.chunk = g->large ? 2 * TC_PACK_CHUNK_LARGE : TC_PACK_CHUNK_SMALL;
    // first[b]: the tensor holding flat position b*chunk, i.e. the last
    // tensor whose offset is <= that position (zero-size tensors at the same
    // offset come before the one that holds it).  The final entry is the
    // tensor holding position N-1.
    auto tensor_at = [&](int64_t j) {
        auto it = std::upper_bound(g->offsets.begin(), g->offsets.begin() + n, j);
        return static_cast<int32_t>(it - g->offsets.begin()) - 1;
    };
    for (tc_chunking* c : {&g->sep, &g->tpack, &g->tpack_fine, &g->pipe, &g->pipe_fine, &g->sep2}) {
        c->nchunks = (g->N + c->chunk - 1) / c->chunk;
        if (c->nchunks > INT32_MAX / 2) { set_error("group too large"); delete g; return nullptr; }
        c->first.resize(static_cast<size_t>(c->nchunks) + 1);
        for (int64_t b = 0; b < c->nchunks; ++b) c->first[b] = tensor_at(b * c->chunk);
        c->first[c->nchunks] = g->N > 0 ? tensor_at(g->N - 1) : 0;
    }
    g->slot_bounds = true;
    for (int32_t t = 1; t < n; ++t)
        if (g->offsets[t] % 4 != 0 && g->offsets[t] < g->N / 4 * 4) g->slot_bounds = false;

    hipError_t e = hipGetDevice(&g->device);
    if (e != hipSuccess) { hip_fail(e, "hipGetDevice"); delete g; return nullptr; }
    size_t ob = g->offsets.size() * sizeof(int64_t);
    if ((e = hipMalloc(&g->d_offsets, ob)) != hipSuccess ||
        (e = hipMemcpy(g->d_offsets, g->offsets.data(), ob, hipMemcpyHostToDevice)) != hipSuccess) {
        hip_fail(e, "group offset table");
        tc_group_destroy(g);
        return nullptr;
    }
    for (tc_chunking* c : {&g->sep, &g->tpack, &g->tpack_fine, &g->pipe, &g->pipe_fine, &g->sep2}) {
        const size_t cb = c->first.size() * sizeof(int32_t);
        if ((e = hipMalloc(&c->d_first, cb)) != hipSuccess ||
            (e = hipMemcpy(c->d_first, c->first.data(), cb, hipMemcpyHostToDevice)) != hipSuccess) {
            hip_fail(e, "group chunk table");
            tc_group_destroy(g);
            return nullptr;
        }
    }
    return g;
}

TC_API void tc_group_destroy(tc_group* g) {
    if (!g) return;
    if (g->d_offsets) (void)hipFree(g->d_offsets);
    for (tc_chunking* c : {&g->sep, &g->tpack, &g->tpack_fine, &g->pipe, &g->pipe_fine, &g->sep2})
        if (c->d_first) (void)hipFree(c->d_first);
    delete g;
}

TC_API int64_t tc_group_numel(const tc_group* g) { return g ? g->N : -1; }

TC_API int32_t tc_group_ntensors(const tc_group* g) { return g ? g->n : -1; }

TC_API int32_t tc_group_offsets(const tc_group* g, int64_t* out) {
    clear_error();
    if (!g || !out) return fail(TC_EINVAL, "tc_group_offsets: NULL argument");
    std::memcpy(out, g->offsets.data(), g->offsets.size() * sizeof(int64_t));
    return TC_OK;
}

// ----------------------------------------------------------- tensor lists

TC_API tc_tensorlist* tc_tensorlist_create(const tc_group* g, int32_t K, const void* const* ptrs,
                                           int32_t dtype) {
    clear_error();
    if (!g || !ptrs) { set_error("tc_tensorlist_create: NULL argument"); return nullptr; }
    if (K < 1 || K > TC_MAX_K) { set_error("K = %d outside [1, %d]", K, TC_MAX_K); return nullptr; }
    const int es = elem_size(dtype);
    if (!es) { set_error("unknown dtype %d", dtype); return nullptr; }
    if (check_device(g) != TC_OK) return nullptr;
    for (int32_t k = 0; k < K; ++k)
        for (int32_t t = 0; t < g->n; ++t) {
            const void* p = ptrs[static_cast<int64_t>(k) * g->n + t];
            if (g->sizes[t] == 0) continue;
            if (!p) { set_error("tensor %d of copy %d is NULL", t, k); return nullptr; }
            if (!aligned(p, es)) { set_error("tensor %d of copy %d is not %d-byte aligned", t, k, es); return nullptr; }
        }
    auto* tl = new (std::nothrow) tc_tensorlist();
    if (!tl) { set_error("out of host memory"); return nullptr; }
    tl->g = g;
    tl->K = K;
    tl->dtype = dtype;
    tl->elem = es;
    tl->ptrs.assign(ptrs, ptrs + static_cast<int64_t>(K) * g->n);
    uintptr_t bits = 0;
    for (int64_t q = 0; q < static_cast<int64_t>(tl->ptrs.size()); ++q)
        if (g->sizes[q % g->n] > 0) bits |= reinterpret_cast<uintptr_t>(tl->ptrs[q]);
    tl->slot_aligned = (bits & static_cast<uintptr_t>(4 * es - 1)) == 0;
    const size_t bytes = tl->ptrs.size() * sizeof(void*);
    hipError_t e = hipMalloc(&tl->d_ptrs, bytes);
    if (e != hipSuccess) { hip_fail(e, "hipMalloc (pointer table)"); delete tl; return nullptr; }
    e = hipMemcpy(tl->d_ptrs, tl->ptrs.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) { hip_fail(e, "hipMemcpy (pointer table)"); tc_tensorlist_destroy(tl); return nullptr; }
    return tl;
}

TC_API void tc_tensorlist_destroy(tc_tensorlist* tl) {
    if (!tl) return;
    if (tl->d_ptrs) (void)hipFree(tl->d_ptrs);
    delete tl;
}

// ------------------------------------------------------------ pack/unpack

static int32_t pack_common(const tc_tensorlist* tl, void* const* flat, bool unpack, void* stream) {
    clear_error();
    if (!tl || !flat) return fail(TC_EINVAL, "NULL argument");
    const tc_group* g = tl->g;
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    bool flat_aligned = true;
    const int64_t bytes = g->N * tl->elem;
    for (int32_t k = 0; k < tl->K; ++k) {
        if (!flat[k]) { set_error("flat[%d] is NULL", k); return TC_EINVAL; }
        if (!aligned(flat[k], tl->elem)) { set_error("flat[%d] is not element-aligned", k); return TC_EINVAL; }
        flat_aligned = flat_aligned && aligned(flat[k], 16);
        for (int32_t q = 0; q < k; ++q)
            if (overlap(flat[k], bytes, flat[q], bytes)) { set_error("flat[%d] overlaps flat[%d]", k, q); return TC_EINVAL; }
    }
    hipError_t e = launch_pack(tl, flat, unpack, flat_aligned, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, unpack ? "tc_unpack launch" : "tc_pack launch");
    return TC_OK;
}

TC_API int32_t tc_pack(const tc_tensorlist* tl, void* const* flat, void* stream) {
    return pack_common(tl, flat, false, stream);
}

TC_API int32_t tc_unpack(const tc_tensorlist* tl, const void* const* flat, void* stream) {
    return pack_common(tl, const_cast<void* const*>(flat), true, stream);
}

// ----------------------------------------------------------------- reduce

TC_API int32_t tc_reduce_ex(const tc_group* g, int32_t K, const void* const* in, int32_t in_dtype,
                            float* out, int32_t op, void* stream) {
    clear_error();
    if (!g) return fail(TC_EINVAL, "group is NULL");
    if (K < 1 || K > TC_MAX_K) { set_error("K = %d outside [1, %d]", K, TC_MAX_K); return TC_EINVAL; }
    if (op != TC_SUM && op != TC_AVG) { set_error("unknown op %d", op); return TC_EINVAL; }
    const int es = elem_size(in_dtype);
    if (!es) { set_error("unknown dtype %d", in_dtype); return TC_EINVAL; }
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    if (!in || !out) return fail(TC_EINVAL, "NULL buffer");
    bool vec = aligned(out, 16);
    if (!aligned(out, 4)) return fail(TC_EINVAL, "out is not 4-byte aligned");
    for (int32_t i = 0; i < K; ++i) {
        if (!in[i]) { set_error("in[%d] is NULL", i); return TC_EINVAL; }
        if (!aligned(in[i], es)) { set_error("in[%d] is not element-aligned", i); return TC_EINVAL; }
        vec = vec && aligned(in[i], es == 4 ? 16 : 8);
        // in place is allowed only as exact identity with a binary32 input:
        // a binary32 output slot covers two bfloat16 input slots, which
        // other lanes read
        if (overlap(in[i], g->N * es, out, g->N * 4) && (in[i] != out || in_dtype != TC_F32)) {
            set_error(in_dtype == TC_F32 ? "out partially overlaps in[%d]"
                                         : "out overlaps in[%d] (no in-place reduction of bfloat16 inputs)", i);
            return TC_EINVAL;
        }
    }
    hipError_t e = launch_reduce(K, in, in_dtype, out, op, g->N, vec, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "tc_reduce launch");
    return TC_OK;
}

TC_API int32_t tc_reduce(const tc_group* g, int32_t K, const float* const* in, float* out, int32_t op,
                         void* stream) {
    return tc_reduce_ex(g, K, reinterpret_cast<const void* const*>(in), TC_F32, out, op, stream);
}

// ------------------------------------------------------------------ easgd

// The step alone (fused false; out and op unused), or fused with the
// reduction of the gradients into out.
static int32_t easgd_common(const tc_group* g, int32_t K, float* const* x, const void* const* grad, int32_t g_dtype,
                            float* x_c, bool fused, float* out, int32_t op, float eta, float rho, void* stream,
                            const char* what) {
    clear_error();
    if (!g) return fail(TC_EINVAL, "group is NULL");
    if (K < 1 || K > TC_MAX_K) { set_error("K = %d outside [1, %d]", K, TC_MAX_K); return TC_EINVAL; }
    const int es = elem_size(g_dtype);
    if (!es) { set_error("unknown dtype %d", g_dtype); return TC_EINVAL; }
    if (fused && op != TC_SUM && op != TC_AVG) { set_error("unknown op %d", op); return TC_EINVAL; }
    if (!std::isfinite(eta) || !std::isfinite(rho)) return fail(TC_EINVAL, "eta and rho must be finite");
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    if (!x || !grad || !x_c || (fused && !out)) return fail(TC_EINVAL, "NULL buffer");
    const int64_t xb = g->N * 4, gb = g->N * es;
    if (!aligned(x_c, 4)) return fail(TC_EINVAL, "x_c is not 4-byte aligned");
    bool vec = aligned(x_c, 16);
    if (out) {
        if (!aligned(out, 4)) return fail(TC_EINVAL, "out is not 4-byte aligned");
        if (overlap(out, xb, x_c, xb)) return fail(TC_EINVAL, "out overlaps x_c");
        vec = vec && aligned(out, 16);
    }
    for (int32_t i = 0; i < K; ++i) {
        if (!x[i] || !grad[i]) { set_error("x[%d] or grad[%d] is NULL", i, i); return TC_EINVAL; }
        if (!aligned(x[i], 4) || !aligned(grad[i], es)) { set_error("x[%d] or grad[%d] misaligned", i, i); return TC_EINVAL; }
        vec = vec && aligned(x[i], 16) && aligned(grad[i], es == 4 ? 16 : 8);
        if (overlap(x[i], xb, x_c, xb)) { set_error("x[%d] overlaps x_c", i); return TC_EINVAL; }
        if (overlap(grad[i], gb, x_c, xb)) { set_error("grad[%d] overlaps x_c", i); return TC_EINVAL; }
        if (out && overlap(out, xb, x[i], xb)) { set_error("out overlaps x[%d]", i); return TC_EINVAL; }
        if (out && overlap(out, xb, grad[i], gb)) { set_error("out overlaps grad[%d]", i); return TC_EINVAL; }
        for (int32_t q = 0; q < K; ++q) {
            if (q < i && overlap(x[i], xb, x[q], xb)) { set_error("x[%d] overlaps x[%d]", i, q); return TC_EINVAL; }
            if (overlap(grad[q], gb, x[i], xb)) { set_error("grad[%d] overlaps x[%d]", q, i); return TC_EINVAL; }
        }
    }
    hipError_t e = launch_easgd(K, x, grad, g_dtype, x_c, out, op, eta, rho, g->N, vec,
                                static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, what);
    return TC_OK;
}

TC_API int32_t easgd_step_ex(const tc_group* g, int32_t K, float* const* x, const void* const* grad,
                             int32_t g_dtype, float* x_c, float eta, float rho, void* stream) {
    return easgd_common(g, K, x, grad, g_dtype, x_c, false, nullptr, TC_SUM, eta, rho, stream, "easgd_step launch");
}

TC_API int32_t reduce_easgd_step(const tc_group* g, int32_t K, float* const* x, const void* const* grad,
                                 int32_t g_dtype, float* x_c, float* out, int32_t op, float eta, float rho,
                                 void* stream) {
    return easgd_common(g, K, x, grad, g_dtype, x_c, true, out, op, eta, rho, stream, "reduce_easgd_step launch");
}

TC_API int32_t easgd_step(const tc_group* g, int32_t K, float* const* x, const float* const* grad, float* x_c,
                          float eta, float rho, void* stream) {
    return easgd_step_ex(g, K, x, reinterpret_cast<const void* const*>(grad), TC_F32, x_c, eta, rho, stream);
}

// ---------------------------------------------------------- tensor layout

TC_API int64_t tc_tensor_numel(const tc_group* g, int32_t K) {
    if (!g || K < 1 || K > TC_MAX_K) return -1;
    return (g->N + 3) / 4 * 4 * K;
}

static int32_t tensor_pack_common(const tc_tensorlist* tl, void* tensor, bool unpack, void* stream) {
    clear_error();
    if (!tl) return fail(TC_EINVAL, "NULL tensor list");
    const tc_group* g = tl->g;
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    if (!tensor) return fail(TC_EINVAL, "tensor is NULL");
    if (!aligned(tensor, 16)) return fail(TC_EINVAL, "tensor buffers must be 16-byte aligned");
    hipError_t e = launch_tensor_pack(tl, tensor, unpack, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, unpack ? "tc_unpack_tensor launch" : "tc_pack_tensor launch");
    return TC_OK;
}

TC_API int32_t tc_pack_tensor(const tc_tensorlist* tl, void* tensor, void* stream) {
    return tensor_pack_common(tl, tensor, false, stream);
}

TC_API int32_t tc_unpack_tensor(const tc_tensorlist* tl, const void* tensor, void* stream) {
    return tensor_pack_common(tl, const_cast<void*>(tensor), true, stream);
}

TC_API int32_t tc_reduce_tensor(const tc_group* g, int32_t K, const void* in, int32_t in_dtype, float* out,
                                int32_t op, void* stream) {
    clear_error();
    if (!g) return fail(TC_EINVAL, "group is NULL");
    if (K < 1 || K > TC_MAX_K) { set_error("K = %d outside [1, %d]", K, TC_MAX_K); return TC_EINVAL; }
    if (op != TC_SUM && op != TC_AVG) { set_error("unknown op %d", op); return TC_EINVAL; }
    const int es = elem_size(in_dtype);
    if (!es) { set_error("unknown dtype %d", in_dtype); return TC_EINVAL; }
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    if (!in || !out) return fail(TC_EINVAL, "NULL buffer");
    if (!aligned(in, 16) || !aligned(out, 16)) return fail(TC_EINVAL, "tensor-layout calls need 16-byte aligned buffers");
    if (overlap(in, tc_tensor_numel(g, K) * es, out, g->N * 4)) return fail(TC_EINVAL, "out overlaps the input tensor");
    hipError_t e = launch_tensor_reduce(K, in, in_dtype, out, op, g->N, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "tc_reduce_tensor launch");
    return TC_OK;
}

// As easgd_common, on tensor-layout buffers.
static int32_t tensor_easgd_common(const tc_group* g, int32_t K, float* x, const void* grad, int32_t g_dtype,
                                   float* x_c, bool fused, float* out, int32_t op, float eta, float rho,
                                   void* stream, const char* what) {
    clear_error();
    if (!g) return fail(TC_EINVAL, "group is NULL");
    if (K < 1 || K > TC_MAX_K) { set_error("K = %d outside [1, %d]", K, TC_MAX_K); return TC_EINVAL; }
    const int es = elem_size(g_dtype);
    if (!es) { set_error("unknown dtype %d", g_dtype); return TC_EINVAL; }
    if (fused && op != TC_SUM && op != TC_AVG) { set_error("unknown op %d", op); return TC_EINVAL; }
    if (!std::isfinite(eta) || !std::isfinite(rho)) return fail(TC_EINVAL, "eta and rho must be finite");
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    if (!x || !grad || !x_c || (fused && !out)) return fail(TC_EINVAL, "NULL buffer");
    if (!aligned(x, 16) || !aligned(grad, 16) || !aligned(x_c, 16) || (out && !aligned(out, 16)))
        return fail(TC_EINVAL, "tensor-layout calls need 16-byte aligned buffers");
    const int64_t tn = tc_tensor_numel(g, K);
    if (overlap(x, tn * 4, grad, tn * es)) return fail(TC_EINVAL, "x overlaps grad");
    if (overlap(x, tn * 4, x_c, g->N * 4)) return fail(TC_EINVAL, "x overlaps x_c");
    if (overlap(grad, tn * es, x_c, g->N * 4)) return fail(TC_EINVAL, "grad overlaps x_c");
    if (out && (overlap(out, g->N * 4, x, tn * 4) || overlap(out, g->N * 4, grad, tn * es) ||
                overlap(out, g->N * 4, x_c, g->N * 4)))
        return fail(TC_EINVAL, "out overlaps x, grad or x_c");
    hipError_t e = launch_tensor_easgd(K, x, grad, g_dtype, x_c, out, op, eta, rho, g->N,
                                       static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, what);
    return TC_OK;
}

TC_API int32_t easgd_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad, int32_t g_dtype,
                                 float* x_c, float eta, float rho, void* stream) {
    return tensor_easgd_common(g, K, x, grad, g_dtype, x_c, false, nullptr, TC_SUM, eta, rho, stream,
                               "easgd_step_tensor launch");
}

TC_API int32_t reduce_easgd_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad, int32_t g_dtype,
                                        float* x_c, float* out, int32_t op, float eta, float rho, void* stream) {
    return tensor_easgd_common(g, K, x, grad, g_dtype, x_c, true, out, op, eta, rho, stream,
                               "reduce_easgd_step_tensor launch");
}

// ------------------------------------------- schedules and synchronous SGD

namespace {

// Shared checks of the separate-buffer step calls: K, finite scalars, the
// device; returns TC_OK or an error (N == 0 is reported as TC_OK by the
// caller before buffers are inspected).
int32_t check_step(const tc_group* g, int32_t K, int32_t g_dtype, float s0, float s1) {
    if (!g) return fail(TC_EINVAL, "group is NULL");
    if (K < 1 || K > TC_MAX_K) { set_error("K = %d outside [1, %d]", K, TC_MAX_K); return TC_EINVAL; }
    if (!elem_size(g_dtype)) { set_error("unknown dtype %d", g_dtype); return TC_EINVAL; }
    if (!std::isfinite(s0) || !std::isfinite(s1)) return fail(TC_EINVAL, "step sizes must be finite");
    return check_device(g);
}

// x[0..K) pairwise disjoint, each 4-byte aligned; *vec &= 16-byte aligned.
int32_t check_workers(const tc_group* g, int32_t K, float* const* x, bool* vec) {
    if (!x) return fail(TC_EINVAL, "NULL buffer array");
    const int64_t xb = g->N * 4;
    for (int32_t i = 0; i < K; ++i) {
        if (!x[i]) { set_error("x[%d] is NULL", i); return TC_EINVAL; }
        if (!aligned(x[i], 4)) { set_error("x[%d] misaligned", i); return TC_EINVAL; }
        *vec = *vec && aligned(x[i], 16);
        for (int32_t q = 0; q < i; ++q)
            if (overlap(x[i], xb, x[q], xb)) { set_error("x[%d] overlaps x[%d]", i, q); return TC_EINVAL; }
    }
    return TC_OK;
}

// grad[0..K) element-aligned and disjoint from every x (and from each other
// when `writable`).
int32_t check_grads(const tc_group* g, int32_t K, const void* const* grad, int es, float* const* x, bool writable,
                    bool* vec) {
    if (!grad) return fail(TC_EINVAL, "NULL buffer array");
    const int64_t gb = g->N * es, xb = g->N * 4;
    for (int32_t i = 0; i < K; ++i) {
        if (!grad[i]) { set_error("grad[%d] is NULL", i); return TC_EINVAL; }
        if (!aligned(grad[i], es)) { set_error("grad[%d] misaligned", i); return TC_EINVAL; }
        *vec = *vec && aligned(grad[i], es == 4 ? 16 : 8);
        for (int32_t q = 0; q < K; ++q) {
            if (overlap(grad[i], gb, x[q], xb)) { set_error("grad[%d] overlaps x[%d]", i, q); return TC_EINVAL; }
            if (writable && q < i && overlap(grad[i], gb, grad[q], gb)) {
                set_error("grad[%d] overlaps grad[%d]", i, q);
                return TC_EINVAL;
            }
        }
    }
    return TC_OK;
}

int32_t launched(hipError_t e, const char* what) { return e == hipSuccess ? TC_OK : hip_fail(e, what); }

int32_t check_tensor_step(const tc_group* g, const void* x, int64_t xbytes, const void* grad, int64_t gbytes) {
    if (!x || (gbytes && !grad)) return fail(TC_EINVAL, "NULL buffer");
    if (!aligned(x, 16) || (gbytes && !aligned(grad, 16)))
        return fail(TC_EINVAL, "tensor-layout calls need 16-byte aligned buffers");
    if (gbytes && overlap(x, xbytes, grad, gbytes)) return fail(TC_EINVAL, "x overlaps grad");
    (void)g;
    return TC_OK;
}

int32_t check_order(int32_t K, const int32_t* order, int32_t R) {
    if (R < 0 || R > K) { set_error("R = %d outside [0, K = %d]", R, K); return TC_EINVAL; }
    if (R && !order) return fail(TC_EINVAL, "order is NULL");
    bool seen[TC_MAX_K] = {};
    for (int32_t r = 0; r < R; ++r) {
        if (order[r] < 0 || order[r] >= K) { set_error("order[%d] = %d outside [0, K)", r, order[r]); return TC_EINVAL; }
        if (seen[order[r]]) { set_error("worker %d exchanges twice", order[r]); return TC_EINVAL; }
        seen[order[r]] = true;
    }
    return TC_OK;
}

}  // namespace

TC_API int32_t sgd_step(const tc_group* g, int32_t K, float* const* x, const void* const* grad, int32_t g_dtype,
                        float eta, void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, g_dtype, eta, 0.0f)) return r;
    if (g->N == 0) return TC_OK;
    bool vec = true;
    if (int32_t r = check_workers(g, K, x, &vec)) return r;
    if (int32_t r = check_grads(g, K, grad, elem_size(g_dtype), x, false, &vec)) return r;
    return launched(launch_sgd(K, x, grad, g_dtype, eta, g->N, vec, static_cast<hipStream_t>(stream)), "sgd_step launch");
}

TC_API int32_t sgd_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad, int32_t g_dtype, float eta,
                               void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, g_dtype, eta, 0.0f)) return r;
    if (g->N == 0) return TC_OK;
    const int64_t tn = tc_tensor_numel(g, K);
    if (int32_t r = check_tensor_step(g, x, tn * 4, grad, tn * elem_size(g_dtype))) return r;
    return launched(launch_tensor_sgd(K, x, grad, g_dtype, eta, g->N, static_cast<hipStream_t>(stream)),
                    "sgd_step_tensor launch");
}

TC_API int32_t easgd_period_step(const tc_group* g, int32_t K, float* const* x, const void* const* grad,
                                 int32_t g_dtype, float* x_c, float eta, float rho, int64_t iteration, int32_t tau,
                                 void* stream) {
    clear_error();
    if (tau < 1 || iteration < 0) { set_error("need tau >= 1 and iteration >= 0"); return TC_EINVAL; }
    if (iteration % tau == 0) return easgd_step_ex(g, K, x, grad, g_dtype, x_c, eta, rho, stream);
    return sgd_step(g, K, x, grad, g_dtype, eta, stream);
}

TC_API int32_t easgd_period_step_tensor(const tc_group* g, int32_t K, float* x, const void* grad, int32_t g_dtype,
                                        float* x_c, float eta, float rho, int64_t iteration, int32_t tau,
                                        void* stream) {
    clear_error();
    if (tau < 1 || iteration < 0) { set_error("need tau >= 1 and iteration >= 0"); return TC_EINVAL; }
    if (iteration % tau == 0) return easgd_step_tensor(g, K, x, grad, g_dtype, x_c, eta, rho, stream);
    return sgd_step_tensor(g, K, x, grad, g_dtype, eta, stream);
}

TC_API int32_t elastic_async(const tc_group* g, int32_t K, float* const* x, float* x_c, const int32_t* order,
                             int32_t R, float alpha, void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, TC_F32, alpha, 0.0f)) return r;
    if (int32_t r = check_order(K, order, R)) return r;
    if (g->N == 0 || R == 0) return TC_OK;
    bool vec = true;
    if (int32_t r = check_workers(g, K, x, &vec)) return r;
    if (!x_c || !aligned(x_c, 4)) return fail(TC_EINVAL, "x_c is NULL or misaligned");
    vec = vec && aligned(x_c, 16);
    for (int32_t i = 0; i < K; ++i)
        if (overlap(x[i], g->N * 4, x_c, g->N * 4)) { set_error("x[%d] overlaps x_c", i); return TC_EINVAL; }
    return launched(launch_elastic_async(K, x, x_c, order, R, alpha, g->N, vec, static_cast<hipStream_t>(stream)),
                    "elastic_async launch");
}

TC_API int32_t elastic_async_tensor(const tc_group* g, int32_t K, float* x, float* x_c, const int32_t* order,
                                    int32_t R, float alpha, void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, TC_F32, alpha, 0.0f)) return r;
    if (int32_t r = check_order(K, order, R)) return r;
    if (g->N == 0 || R == 0) return TC_OK;
    const int64_t tn = tc_tensor_numel(g, K);
    if (int32_t r = check_tensor_step(g, x, tn * 4, x_c, g->N * 4)) return r;
    return launched(launch_tensor_elastic_async(K, x, x_c, order, R, alpha, g->N, static_cast<hipStream_t>(stream)),
                    "elastic_async_tensor launch");
}

TC_API int32_t sync_sgd_step(const tc_group* g, int32_t K, float* const* x, void* const* grad, int32_t g_dtype,
                             float eta, float rescale, int32_t broadcast, void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, g_dtype, eta, rescale)) return r;
    if (broadcast && g_dtype != TC_F32)
        return fail(TC_EUNSUPPORTED, "broadcasting the summed gradient needs binary32 gradients");
    if (g->N == 0) return TC_OK;
    bool vec = true;
    if (int32_t r = check_workers(g, K, x, &vec)) return r;
    if (int32_t r = check_grads(g, K, const_cast<const void* const*>(grad), elem_size(g_dtype), x, broadcast != 0, &vec))
        return r;
    return launched(launch_sync_sgd(K, x, grad, g_dtype, eta, rescale, broadcast, g->N, vec,
                                    static_cast<hipStream_t>(stream)),
                    "sync_sgd_step launch");
}

TC_API int32_t sync_sgd_step_tensor(const tc_group* g, int32_t K, float* x, void* grad, int32_t g_dtype, float eta,
                                    float rescale, int32_t broadcast, void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, g_dtype, eta, rescale)) return r;
    if (broadcast && g_dtype != TC_F32)
        return fail(TC_EUNSUPPORTED, "broadcasting the summed gradient needs binary32 gradients");
    if (g->N == 0) return TC_OK;
    const int64_t tn = tc_tensor_numel(g, K);
    if (int32_t r = check_tensor_step(g, x, tn * 4, grad, tn * elem_size(g_dtype))) return r;
    return launched(launch_tensor_sync_sgd(K, x, grad, g_dtype, eta, rescale, broadcast, g->N,
                                           static_cast<hipStream_t>(stream)),
                    "sync_sgd_step_tensor launch");
}

TC_API int32_t tc_broadcast(const tc_group* g, int32_t K, const void* src, void* const* dst, int32_t dtype,
                            void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, dtype, 0.0f, 0.0f)) return r;
    if (g->N == 0) return TC_OK;
    const int es = elem_size(dtype);
    const int64_t b = g->N * es;
    if (!src || !dst) return fail(TC_EINVAL, "NULL buffer");
    if (!aligned(src, es)) return fail(TC_EINVAL, "src misaligned");
    bool vec = aligned(src, 16);
    for (int32_t i = 0; i < K; ++i) {
        if (!dst[i] || !aligned(dst[i], es)) { set_error("dst[%d] is NULL or misaligned", i); return TC_EINVAL; }
        vec = vec && aligned(dst[i], 16);
        if (overlap(dst[i], b, src, b)) { set_error("dst[%d] overlaps src", i); return TC_EINVAL; }
        for (int32_t q = 0; q < i; ++q)
            if (overlap(dst[i], b, dst[q], b)) { set_error("dst[%d] overlaps dst[%d]", i, q); return TC_EINVAL; }
    }
    return launched(launch_broadcast(K, src, dst, es, g->N, vec, static_cast<hipStream_t>(stream)), "tc_broadcast launch");
}

TC_API int32_t tc_broadcast_tensor(const tc_group* g, int32_t K, const void* src, void* dst, int32_t dtype,
                                   void* stream) {
    clear_error();
    if (int32_t r = check_step(g, K, dtype, 0.0f, 0.0f)) return r;
    if (g->N == 0) return TC_OK;
    const int es = elem_size(dtype);
    if (!src || !dst) return fail(TC_EINVAL, "NULL buffer");
    if (!aligned(src, 16) || !aligned(dst, 16)) return fail(TC_EINVAL, "tensor-layout calls need 16-byte aligned buffers");
    if (overlap(dst, tc_tensor_numel(g, K) * es, src, g->N * es)) return fail(TC_EINVAL, "dst overlaps src");
    return launched(launch_tensor_broadcast(K, src, dst, es, g->N, static_cast<hipStream_t>(stream)),
                    "tc_broadcast_tensor launch");
}

// ------------------------------------------------------------ pipeline

TC_API int32_t easgd_pipeline_tensor(const tc_tensorlist* grads, const tc_tensorlist* params, void* g_tensor,
                                     float* gbar, float* x, float* x_c, float eta, float rho, void* stream) {
    clear_error();
    if (!grads || !params) return fail(TC_EINVAL, "NULL tensor list");
    const tc_group* g = grads->g;
    if (params->g != g) return fail(TC_EINVAL, "the gradient and parameter lists belong to different groups");
    if (params->K != grads->K) return fail(TC_EINVAL, "the gradient and parameter lists have different K");
    if (params->dtype != TC_F32) return fail(TC_EINVAL, "parameter tensors must be binary32");
    if (!std::isfinite(eta) || !std::isfinite(rho)) return fail(TC_EINVAL, "eta and rho must be finite");
    if (int32_t r = check_device(g)) return r;
    if (g->N == 0) return TC_OK;
    if (!gbar || !x || !x_c) return fail(TC_EINVAL, "NULL buffer");
    if (!aligned(gbar, 16) || !aligned(x, 16) || !aligned(x_c, 16) || (g_tensor && !aligned(g_tensor, 16)))
        return fail(TC_EINVAL, "tensor-layout calls need 16-byte aligned buffers");
    const int K = grads->K;
    const int64_t tn = tc_tensor_numel(g, K), nb = g->N * 4;
    const int64_t gtb = g_tensor ? tn * grads->elem : 0;
    if (overlap(x, tn * 4, x_c, nb)) return fail(TC_EINVAL, "x overlaps x_c");
    if (overlap(x, tn * 4, gbar, nb)) return fail(TC_EINVAL, "x overlaps gbar");
    if (overlap(x_c, nb, gbar, nb)) return fail(TC_EINVAL, "x_c overlaps gbar");
    if (gtb && (overlap(g_tensor, gtb, x, tn * 4) || overlap(g_tensor, gtb, x_c, nb) || overlap(g_tensor, gtb, gbar, nb)))
        return fail(TC_EINVAL, "g_tensor overlaps another buffer");
    return launched(launch_tensor_pipeline(grads, params, g_tensor, gbar, x, x_c, eta, rho,
                                           static_cast<hipStream_t>(stream)),
                    "easgd_pipeline_tensor launch");
}
