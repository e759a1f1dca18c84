// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "tc.h"

#define TC_API extern "C" __attribute__((visibility("default")))

namespace tc {

// Elements per chunk: one workgroup takes one chunk (of one copy, on
// separate buffers; of all K copies, on the tensor layout).  Each kind of
// kernel cuts the group its own way, chosen from the group's mean tensor
// size (measured on MI355X):
// - separate-buffer pack/unpack: groups of large tensors (almost every chunk
//   inside one tensor) move best in short chunks that a workgroup covers in
//   one batch per lane; groups of many small tensors in longer chunks, which
//   spread the per-chunk segment staging over more data (4,096: pack plus
//   unpack 4% faster than with 8,192, 10% faster than with 2,048), and
//   2-byte elements on groups of large tensors in chunks of twice the
//   elements (the bytes of a binary32 chunk);
// - tensor-layout pack/unpack, whose workgroups move all K copies of a chunk:
//   1,024 elements (against 2,048 and 512 on VGG-16's straight path, and
//   against 512 and 2,048 to 8,192 on 10,000 small tensors), but 512 through
//   the tiles for unpack on large-tensor groups (ResNet-50 K = 8 +4-5%) or
//   with copy groups, and for pack from K = 12 (3-9% slower at K <= 8); and
//   the separate-buffer chunks at P <= 2 (but the direct binary32 unpack at
//   P = 2), where 1,024 elements move only 4-16 KB;
// - the pipelined step: 512 elements (7-8% faster than 2,048 on ResNet-50,
//   VGG-16 and 10,000 small tensors; 2% faster than 1,024 on the latter),
//   but the tensor-layout pack's 1,024 at P = 1, and at P = 2 except for
//   binary32 gradients on the straight path, and 256 on groups of large
//   tensors from K = 8 (+2.5-7% there).
// All are multiples of every vector width (4, 8).
#ifndef TC_PACK_CHUNK_LARGE
#define TC_PACK_CHUNK_LARGE 2048
#endif
#ifndef TC_PACK_CHUNK_SMALL
#define TC_PACK_CHUNK_SMALL 4096
#endif
#ifndef TC_TPACK_CHUNK
#define TC_TPACK_CHUNK 1024
#endif
#ifndef TC_TPACK_CHUNK_FINE
#define TC_TPACK_CHUNK_FINE 512
#endif
#ifndef TC_PIPE_CHUNK
#define TC_PIPE_CHUNK 512
#endif
#ifndef TC_PIPE_CHUNK_FINE
#define TC_PIPE_CHUNK_FINE 256
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

// A load or store at an address with no alignment beyond the element size:
// on gfx950 global memory is accessed in unaligned mode, so a 16-byte (or
// 8-byte) access at any byte address is one vector instruction, which the
// memory pipeline splits over the cache lines it touches.
template <typename V>
__device__ __forceinline__ V gld_u(uintptr_t a) {
    typedef V Vu __attribute__((aligned(1)));
    return *reinterpret_cast<const TC_GLOBAL Vu*>(a);
}
template <typename V>
__device__ __forceinline__ void gst_u(uintptr_t a, V v) {
    typedef V Vu __attribute__((aligned(1)));
    *reinterpret_cast<TC_GLOBAL Vu*>(a) = v;
}

// Workgroup w of a launch runs on XCD w % 8, and each of the 8 XCDs has its
// own L2 cache and address-translation caches.  tile_of<R> renumbers the
// workgroups so that, within every 8R consecutive tiles, each XCD takes R
// consecutive tiles (R = 1: no renumbering; a last partial group of 8R
// tiles keeps its order).  The tensor-layout reduction, step and broadcast
// kernels take R = 128 (runs of 128 tiles of 32 to 128 slots): measured on
// MI355X against R = 1, the fused step +2.5% (VGG-16, K = 4), +5% (ResNet-50,
// K = 8) and +3.6% (10,000 tensors, K = 16), the reduction +2 to +4%; R = 32
// to 512 gain less or the same.  The pack, unpack and pipelined kernels,
// whose workgroups stage segment tables, and the separate-buffer kernels
// measured level or slower with any R, and keep their order.
#ifndef TC_XCD_RUN_STEP
#define TC_XCD_RUN_STEP 128
#endif
template <int R>
__device__ __forceinline__ uint32_t tile_of(uint32_t b, uint32_t nb) {
    if constexpr (R <= 1) {
        return b;
    } else {
        constexpr uint32_t S = 8u * R;
        if (b >= nb / S * S) return b;
        return b / S * S + (b % 8u) * R + (b / 8u) % R;
    }
}

// A tensor's start relative to a chunk's first element, clamped to the
// chunk [0, clen]: the chunk-relative segment bounds the pack, unpack and
// pipelined kernels stage.
__device__ __forceinline__ int32_t clamp_rel(int64_t v, int32_t clen) {
    return static_cast<int32_t>(v < 0 ? 0 : (v > clen ? clen : v));
}

// Records a printf-style message as this thread's last error.
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

// Launchers, defined next to their kernels.  Arguments are validated by the
// caller; these only pick a kernel and enqueue it on `stream`.
hipError_t launch_reduce(int K, const void* const* in, int in_dtype, float* out, int op,
                         int64_t n, bool vector_ok, hipStream_t stream);
// out == nullptr: the step alone; otherwise the step fused with the
// reduction of the gradients into out (op TC_SUM or TC_AVG).
hipError_t launch_easgd(int K, float* const* x, const void* const* g, int g_dtype, float* xc, float* out, int op,
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
hipError_t launch_tensor_easgd(int K, float* x, const void* g, int g_dtype, float* xc, float* out, int op, float eta,
                               float rho, int64_t n, hipStream_t stream);
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

// One cut of the flat index space into chunks of `chunk` elements (the last
// one shorter) with, per chunk, the first tensor it touches.
struct tc_chunking {
    int64_t chunk = 0;           // elements per chunk
    int64_t nchunks = 0;         // ceil(N / chunk)
    std::vector<int32_t> first;  // nchunks + 1
    int32_t* d_first = nullptr;  // device copy
};

// Group descriptor: host copies of sizes and offsets, and device copies of
// the offset table and of each chunking's first-segment table.
struct tc_group {
    int32_t n = 0;
    int64_t N = 0;
    int device = 0;
    std::vector<int64_t> sizes;
    std::vector<int64_t> offsets;  // n + 1
    bool large = false;            // mean tensor size >= TC_PACK_LARGE_MEAN
    tc_chunking sep;               // separate-buffer pack/unpack
    tc_chunking tpack;             // tensor-layout pack/unpack
    tc_chunking tpack_fine;        // tensor-layout pack/unpack through the tiles, where shorter chunks pay
    tc_chunking pipe;              // the pipelined step
    tc_chunking pipe_fine;         // the pipelined step, shorter chunks
    tc_chunking sep2;              // separate-buffer pack/unpack, 2-byte elements
    bool slot_bounds = false;      // every tensor boundary before the last,
                                   // partial slot is a multiple of 4
    int64_t* d_offsets = nullptr;
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
