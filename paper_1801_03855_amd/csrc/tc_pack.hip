// Pack / unpack between K copies of a group's separate tensors and the
// copies' flat buffers, in one launch for all tensors and all copies.
//
// The flat index space is cut into chunks of kChunk elements; workgroup
// (b, k) copies chunk b of copy k.  The host precomputed, for every chunk,
// the first tensor it touches; the workgroup stages the offsets (relative to
// the chunk, clamped to it) and pointers of the tensors overlapping its
// chunk in LDS, so a group of thousands of small tensors costs one launch
// and one table read per workgroup.  Each lane then owns 16-byte slots of
// the flat side (coalesced 1 KiB per wave instruction), finds the tensor
// holding the slot by binary search in LDS, and moves the slot with one
// 16-byte access when it lies inside one tensor at a 16-byte aligned
// address there, element by element otherwise (tensor boundaries, tensors
// whose data is not 16-byte aligned, the ragged end of the group).  A chunk
// touching more than kMaxStage tensors (only possible with many tiny or
// empty tensors) searches the device tables in global memory instead.
#include "tc_internal.h"

#ifndef TC_PACK_THREADS
#define TC_PACK_THREADS 256
#endif

namespace tc {
namespace {

typedef unsigned int u4 __attribute__((ext_vector_type(4)));

struct PackKernelArgs {
    const int64_t* offsets;
    const int32_t* chunk_first;
    void* const* ptrs;  // K*n device pointers, copy-major
    int32_t n;
    int64_t N;
    void* flat[TC_MAX_K];
};

// Segment tables: relative offsets rel(0..nseg) (clamped to [0, clen]), the
// true start of segment 0 relative to the chunk (<= 0), pointers ptr(s).
struct LdsTable {
    const int32_t* rel;
    void* const* ptr;
    __device__ int32_t r(int s) const { return rel[s]; }
    __device__ void* p(int s) const { return ptr[s]; }
};

struct GlobalTable {
    const int64_t* off;  // offsets + lo
    void* const* ptr;    // copy's pointers + lo
    int64_t cstart;
    int32_t clen;
    __device__ int32_t r(int s) const {
        int64_t v = off[s] - cstart;
        return static_cast<int32_t>(v < 0 ? 0 : (v > clen ? clen : v));
    }
    __device__ void* p(int s) const { return ptr[s]; }
};

template <typename T, bool UNPACK, bool FLAT16, typename Table>
__device__ __forceinline__ void copy_chunk(const Table& tab, int nseg, int64_t first_start, int32_t clen,
                                           T* flat_chunk) {
    constexpr int VEC = 16 / sizeof(T);
    const int nvec = (clen + VEC - 1) / VEC;
    for (int v = threadIdx.x; v < nvec; v += TC_PACK_THREADS) {
        const int jr = v * VEC;
        // last segment whose start is <= jr (rel(0) == 0 always qualifies)
        int lo = 0, hi = nseg - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (tab.r(mid) <= jr) lo = mid; else hi = mid - 1;
        }
        int s = lo;
        int64_t start = s == 0 ? first_start : tab.r(s);
        T* tp = static_cast<T*>(tab.p(s)) + (jr - start);
        if (FLAT16 && jr + VEC <= tab.r(s + 1) &&
            (reinterpret_cast<uintptr_t>(tp) & 15) == 0) {
            u4* fv = reinterpret_cast<u4*>(flat_chunk + jr);
            u4* tv = reinterpret_cast<u4*>(tp);
            if (UNPACK) __builtin_nontemporal_store(__builtin_nontemporal_load(fv), tv);
            else __builtin_nontemporal_store(__builtin_nontemporal_load(tv), fv);
            continue;
        }
        const int cnt = clen - jr < VEC ? clen - jr : VEC;
        for (int q = 0; q < cnt; ++q) {
            const int jq = jr + q;
            while (jq >= tab.r(s + 1)) {
                ++s;
                start = tab.r(s);
            }
            T* te = static_cast<T*>(tab.p(s)) + (jq - start);
            if (UNPACK) *te = flat_chunk[jq];
            else flat_chunk[jq] = *te;
        }
    }
}

template <typename T, bool UNPACK, bool FLAT16>
__global__ __launch_bounds__(TC_PACK_THREADS) void pack_kernel(PackKernelArgs a) {
    __shared__ int32_t s_rel[kMaxStage + 1];
    __shared__ void* s_ptr[kMaxStage];
    const int64_t b = blockIdx.x;
    const int k = blockIdx.y;
    const int64_t cstart = b * kChunk;
    const int32_t clen = static_cast<int32_t>(a.N - cstart < kChunk ? a.N - cstart : kChunk);
    const int32_t lo = a.chunk_first[b];
    const int32_t hi = a.chunk_first[b + 1];
    const int nseg = hi - lo + 1;
    void* const* cp = a.ptrs + static_cast<int64_t>(k) * a.n + lo;
    const int64_t first_start = a.offsets[lo] - cstart;
    T* flat_chunk = static_cast<T*>(a.flat[k]) + cstart;
    if (nseg <= kMaxStage) {
        for (int s = threadIdx.x; s <= nseg; s += TC_PACK_THREADS) {
            int64_t v = a.offsets[lo + s] - cstart;
            s_rel[s] = static_cast<int32_t>(v < 0 ? 0 : (v > clen ? clen : v));
            if (s < nseg) s_ptr[s] = cp[s];
        }
        __syncthreads();
        copy_chunk<T, UNPACK, FLAT16>(LdsTable{s_rel, s_ptr}, nseg, first_start, clen, flat_chunk);
    } else {
        copy_chunk<T, UNPACK, FLAT16>(GlobalTable{a.offsets + lo, cp, cstart, clen}, nseg, first_start, clen,
                                      flat_chunk);
    }
}

template <typename T, bool UNPACK>
hipError_t run(const PackKernelArgs& a, int K, int64_t nchunks, bool flat16, hipStream_t s) {
    dim3 grid(static_cast<unsigned>(nchunks), static_cast<unsigned>(K));
    if (flat16)
        hipLaunchKernelGGL((pack_kernel<T, UNPACK, true>), grid, dim3(TC_PACK_THREADS), 0, s, a);
    else
        hipLaunchKernelGGL((pack_kernel<T, UNPACK, false>), grid, dim3(TC_PACK_THREADS), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pack(const tc_tensorlist* tl, void* const* flat, bool unpack, bool flat_aligned,
                       hipStream_t stream) {
    const tc_group* g = tl->g;
    PackKernelArgs a{};
    a.offsets = g->d_offsets;
    a.chunk_first = g->d_chunk_first;
    a.ptrs = tl->d_ptrs;
    a.n = g->n;
    a.N = g->N;
    for (int k = 0; k < tl->K; ++k) a.flat[k] = flat[k];
    if (tl->elem == 2)
        return unpack ? run<uint16_t, true>(a, tl->K, g->nchunks, flat_aligned, stream)
                      : run<uint16_t, false>(a, tl->K, g->nchunks, flat_aligned, stream);
    return unpack ? run<uint32_t, true>(a, tl->K, g->nchunks, flat_aligned, stream)
                  : run<uint32_t, false>(a, tl->K, g->nchunks, flat_aligned, stream);
}

}  // namespace tc
