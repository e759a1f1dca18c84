// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "tc.h"

#define TC_API extern "C" __attribute__((visibility("default")))

namespace tc {

// Elements per pack/unpack chunk; one workgroup gathers or scatters one
// chunk of one copy.  Chosen per group from its mean tensor size: groups of
// large tensors (almost every chunk inside one tensor) move best in short
// chunks that a workgroup covers in one batch per lane; groups of many small
// tensors in long chunks, which spread the per-chunk segment staging over
// more data (measured on MI355X).  Multiples of every vector width (4, 8).
#ifndef TC_PACK_CHUNK_LARGE
#define TC_PACK_CHUNK_LARGE 2048
#endif
#ifndef TC_PACK_CHUNK_SMALL
#define TC_PACK_CHUNK_SMALL 8192
#endif
#ifndef TC_PACK_LARGE_MEAN
#define TC_PACK_LARGE_MEAN 32768
#endif

// Segments (tensors overlapping one chunk) whose offsets and pointers a
// workgroup stages in LDS; chunks touching more tensors search the global
// tables instead.
constexpr int kMaxStage = 1024;

// Device access to global memory at an address held as an integer (pointers
// read from the tensor lists' tables, addresses formed by arithmetic).  The
// address space is stated so that the compiler emits global, not flat,
// instructions: a flat access also counts against the LDS wait counter, so
// every later wait for an LDS access would wait for it as well.
#define TC_GLOBAL __attribute__((address_space(1)))
template <typename V>
__device__ __forceinline__ V gld(uintptr_t a) {
    return *reinterpret_cast<const TC_GLOBAL V*>(a);
}
template <typename V>
__device__ __forceinline__ V gld_nt(uintptr_t a) {
    return __builtin_nontemporal_load(reinterpret_cast<const TC_GLOBAL V*>(a));
}
template <typename V>
__device__ __forceinline__ void gst(uintptr_t a, V v) {
    *reinterpret_cast<TC_GLOBAL V*>(a) = v;
}
template <typename V>
__device__ __forceinline__ void gst_nt(uintptr_t a, V v) {
    __builtin_nontemporal_store(v, reinterpret_cast<TC_GLOBAL V*>(a));
}

// Records a printf-style message as this thread's last error.
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

// Launchers, defined next to their kernels.  Arguments are validated by the
// caller; these only pick a kernel and enqueue it on `stream`.
hipError_t launch_reduce(int K, const void* const* in, int in_dtype, float* out, int op,
                         int64_t n, bool vector_ok, hipStream_t stream);
hipError_t launch_easgd(int K, float* const* x, const void* const* g, int g_dtype, float* xc,
                        float eta, float rho, int64_t n, bool vector_ok, hipStream_t stream);

hipError_t launch_sgd(int K, float* const* x, const void* const* g, int g_dtype, float eta, int64_t n, bool vector_ok,
                      hipStream_t stream);
hipError_t launch_sync_sgd(int K, float* const* x, void* const* g, int g_dtype, float eta, float rescale, int broadcast,
                           int64_t n, bool vector_ok, hipStream_t stream);
hipError_t launch_elastic_async(int K, float* const* x, float* xc, const int32_t* order, int R, float alpha,
                                int64_t n, bool vector_ok, hipStream_t stream);
hipError_t launch_broadcast(int K, const void* src, void* const* dst, int es, int64_t n, bool vector_ok,
                            hipStream_t stream);

hipError_t launch_pack(const tc_tensorlist* tl, void* const* flat, bool unpack, bool flat_aligned,
                       hipStream_t stream);

// Tensor layout (K copies interleaved in slots of 4 elements).
hipError_t launch_tensor_reduce(int K, const void* in, int in_dtype, float* out, int op, int64_t n,
                                hipStream_t stream);
hipError_t launch_tensor_easgd(int K, float* x, const void* g, int g_dtype, float* xc, float eta, float rho,
                               int64_t n, hipStream_t stream);
hipError_t launch_tensor_pack(const tc_tensorlist* tl, void* tensor, bool unpack, hipStream_t stream);
hipError_t launch_tensor_sgd(int K, float* x, const void* g, int g_dtype, float eta, int64_t n, hipStream_t s);
hipError_t launch_tensor_sync_sgd(int K, float* x, void* g, int g_dtype, float eta, float rescale, int broadcast,
                                  int64_t n, hipStream_t s);
hipError_t launch_tensor_elastic_async(int K, float* x, float* xc, const int32_t* order, int R, float alpha, int64_t n,
                                       hipStream_t s);
hipError_t launch_tensor_broadcast(int K, const void* src, void* dst, int es, int64_t n, hipStream_t s);
hipError_t launch_tensor_pipeline(const tc_tensorlist* grads, const tc_tensorlist* params, void* gt, float* gbar,
                                  float* x, float* xc, float eta, float rho, hipStream_t stream);

}  // namespace tc

// Group descriptor: host copies of sizes and offsets, and device copies of
// the offset table and of the per-chunk first-segment table.
struct tc_group {
    int32_t n = 0;
    int64_t N = 0;
    int device = 0;
    std::vector<int64_t> sizes;
    std::vector<int64_t> offsets;      // n + 1
    int64_t chunk = 0;                 // elements per pack/unpack chunk
    int64_t nchunks = 0;               // ceil(N / chunk)
    std::vector<int32_t> chunk_first;  // nchunks + 1
    bool slot_bounds = false;          // every tensor boundary before the last,
                                       // partial slot is a multiple of 4
    int64_t* d_offsets = nullptr;
    int32_t* d_chunk_first = nullptr;
};

// K copies of a group held as separate tensors: device table of K*n
// pointers, copy-major.
struct tc_tensorlist {
    const tc_group* g = nullptr;
    int32_t K = 0;
    int32_t dtype = TC_F32;
    int32_t elem = 4;
    std::vector<const void*> ptrs;
    bool slot_aligned = false;  // every non-empty tensor starts on a 4-element boundary
    void** d_ptrs = nullptr;
};
