// Pack / unpack between K copies of a group's separate tensors and the
// copies' flat buffers, in one launch for all tensors and all copies.
//
// The flat index space is cut into chunks (of the group's chunk length); workgroup
// (b, k) moves chunk b of copy k.  The host precomputed, for every chunk,
// the first tensor it touches, so the workgroup reads one table entry and
// stages the chunk-relative offsets and pointers of the tensors overlapping
// its chunk (its "segments") in LDS: a group of thousands of small tensors
// costs one launch.
//
// Work is enumerated over 16-byte aligned granules of the destination side
// (the flat buffer for pack, the tensors for unpack): a prefix sum over the
// segments' granule counts, in LDS, lets each lane find its granule by
// binary search.  A granule lying wholly inside one segment is written with
// one 16-byte store; its 16 source bytes are read with one 16-byte load,
// an unaligned one when they do not start on a 16-byte boundary (gfx950
// accesses global memory in unaligned mode).  Granules cut by a
// segment's ends are copied element by element.  So tensors at any element
// alignment, and any flat offset, move with full-width accesses.
//
// A chunk touching more than kMaxStage tensors (only possible with many
// tiny or empty tensors) is copied element by element, searching the device
// tables in global memory.
#include "tc_internal.h"

#ifndef TC_PACK_THREADS
#define TC_PACK_THREADS 256
#endif
// Granules a lane moves at a time: their loads are all issued before the
// first store.
#ifndef TC_PACK_BATCH
#define TC_PACK_BATCH 2
#endif

namespace tc {
namespace {

typedef unsigned int u4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = TC_PACK_THREADS / 64;

struct PackKernelArgs {
    const int64_t* offsets;
    const int32_t* chunk_first;
    void* const* ptrs;  // K*n device pointers, copy-major
    int32_t n;
    int64_t N;
    int64_t chunk;
    void* flat[TC_MAX_K];
};

// Destination byte range [d0, d1) of one segment's part of the chunk, and
// the displacement from a destination byte to its source byte.
struct SegView {
    uintptr_t d0, d1;
    intptr_t delta;
};

template <typename T, bool UNPACK>
__device__ __forceinline__ SegView seg_view(const int32_t* rel, const char* const* ptr, int s,
                                            int64_t first_start, uintptr_t flat0) {
    constexpr intptr_t es = sizeof(T);
    const int32_t e0 = rel[s], e1 = rel[s + 1];
    const int64_t start = s == 0 ? first_start : rel[s];
    // byte address, in the tensor, of chunk-relative flat element 0
    const uintptr_t tens0 = reinterpret_cast<uintptr_t>(ptr[s]) - static_cast<uintptr_t>(start * es);
    SegView v;
    if (UNPACK) {
        v.d0 = tens0 + e0 * es;
        v.d1 = tens0 + e1 * es;
        v.delta = static_cast<intptr_t>(flat0 - tens0);
    } else {
        v.d0 = flat0 + e0 * es;
        v.d1 = flat0 + e1 * es;
        v.delta = static_cast<intptr_t>(tens0 - flat0);
    }
    return v;
}

__device__ __forceinline__ int32_t granules(const SegView& v) {
    if (v.d1 <= v.d0) return 0;
    return static_cast<int32_t>(((v.d1 + 15) >> 4) - (v.d0 >> 4));
}

// Whether destination granule A of segment v is whole (all 16 bytes inside
// the segment's destination range).
__device__ __forceinline__ bool whole(const SegView& v, uintptr_t A) { return A >= v.d0 && A + 16 <= v.d1; }

// The 16 source bytes of a whole granule: one load, non-temporal when they
// are aligned, else one unaligned (cacheable) access (measured on MI355X
// against two aligned loads and a funnel shift: the 10,000-tensor bfloat16
// group at K = 16 packs 6.4% and unpacks 2.6% faster).
__device__ __forceinline__ u4 load_granule(const SegView& v, uintptr_t A) {
    const uintptr_t S = A + v.delta;
    if ((S & 15) == 0) return gld_nt<u4>(S);
    return gld_u<u4>(S);
}

// Element-by-element copy of the part of granule A inside segment v.
template <typename T>
__device__ __forceinline__ void copy_partial(const SegView& v, uintptr_t A) {
    constexpr uintptr_t es = sizeof(T);
    const uintptr_t lo = A > v.d0 ? A : v.d0;
    const uintptr_t hi = A + 16 < v.d1 ? A + 16 : v.d1;
    for (uintptr_t x = lo; x < hi; x += es)
        gst<T>(x, gld<T>(x + v.delta));
}

// Element-by-element copy of a chunk whose segments stay in global memory.
template <typename T, bool UNPACK>
__device__ void copy_chunk_global(const int64_t* off, void* const* cp, int nseg, int64_t cstart, int32_t clen,
                                  T* flat_chunk) {
    for (int jr = threadIdx.x; jr < clen; jr += TC_PACK_THREADS) {
        int lo = 0, hi = nseg - 1;  // last segment whose start is <= jr
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (clamp_rel(off[mid] - cstart, clen) <= jr) lo = mid; else hi = mid - 1;
        }
        const uintptr_t te = reinterpret_cast<uintptr_t>(cp[lo]) + static_cast<uintptr_t>((cstart + jr - off[lo]) * sizeof(T));
        const uintptr_t tf = reinterpret_cast<uintptr_t>(flat_chunk + jr);
        if (UNPACK) gst<T>(te, gld<T>(tf));
        else gst<T>(tf, gld<T>(te));
    }
}

template <typename T, bool UNPACK>
__global__ __launch_bounds__(TC_PACK_THREADS) void pack_kernel(PackKernelArgs a) {
    __shared__ int32_t s_rel[kMaxStage + 1];
    __shared__ const char* s_ptr[kMaxStage];
    __shared__ int32_t s_pre[kMaxStage + 1];
    __shared__ int32_t s_wave[kWaves];
    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int k = blockIdx.y;
    const int64_t cstart = b * a.chunk;
    const int32_t clen = static_cast<int32_t>(a.N - cstart < a.chunk ? a.N - cstart : a.chunk);
    const int32_t lo = a.chunk_first[b];
    const int32_t hi = a.chunk_first[b + 1];
    const int nseg = hi - lo + 1;
    void* const* cp = a.ptrs + static_cast<int64_t>(k) * a.n + lo;
    T* flat_chunk = static_cast<T*>(a.flat[k]) + cstart;
    if (nseg > kMaxStage) {
        copy_chunk_global<T, UNPACK>(a.offsets + lo, cp, nseg, cstart, clen, flat_chunk);
        return;
    }
    const int64_t first_start = a.offsets[lo] - cstart;
    for (int s = tid; s <= nseg; s += TC_PACK_THREADS) {
        s_rel[s] = clamp_rel(a.offsets[lo + s] - cstart, clen);
        if (s < nseg) s_ptr[s] = static_cast<const char*>(cp[s]);
    }
    __syncthreads();

    // exclusive prefix sum of the segments' granule counts (a chunk inside
    // one tensor, the common case for large tensors, needs none)
    const uintptr_t flat0 = reinterpret_cast<uintptr_t>(flat_chunk);
    int total;
    if (nseg == 1) {
        total = granules(seg_view<T, UNPACK>(s_rel, s_ptr, 0, first_start, flat0));
    } else {
        const int spt = (nseg + TC_PACK_THREADS - 1) / TC_PACK_THREADS;
        int local = 0;
        for (int i = 0; i < spt; ++i) {
            const int s = tid * spt + i;
            if (s < nseg) local += granules(seg_view<T, UNPACK>(s_rel, s_ptr, s, first_start, flat0));
        }
        const int lane = tid & 63, wid = tid >> 6;
        int incl = local;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int o = __shfl_up(incl, d, 64);
            if (lane >= d) incl += o;
        }
        if (lane == 63) s_wave[wid] = incl;
        __syncthreads();
        int base = 0;
        total = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            base += w < wid ? s_wave[w] : 0;
            total += s_wave[w];
        }
        int run = base + incl - local;
        for (int i = 0; i < spt; ++i) {
            const int s = tid * spt + i;
            if (s < nseg) {
                s_pre[s] = run;
                run += granules(seg_view<T, UNPACK>(s_rel, s_ptr, s, first_start, flat0));
            }
        }
        __syncthreads();
    }

    constexpr int B = TC_PACK_BATCH;
    for (int q0 = tid; q0 < total; q0 += TC_PACK_THREADS * B) {
        SegView v[B];
        uintptr_t A[B];
        bool full[B];
        u4 val[B];
#pragma unroll
        for (int i = 0; i < B; ++i) {
            const int q = q0 + i * TC_PACK_THREADS;
            full[i] = false;
            if (q < total) {
                int l = 0, h = nseg - 1;  // last segment whose prefix is <= q
                while (l < h) {
                    const int mid = (l + h + 1) >> 1;
                    if (s_pre[mid] <= q) l = mid; else h = mid - 1;
                }
                v[i] = seg_view<T, UNPACK>(s_rel, s_ptr, l, first_start, flat0);
                const int pre = l == 0 ? 0 : s_pre[l];  // the first segment's prefix is 0
                A[i] = ((v[i].d0 >> 4) + static_cast<uintptr_t>(q - pre)) << 4;
                full[i] = whole(v[i], A[i]);
                if (full[i]) val[i] = load_granule(v[i], A[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < B; ++i)
            if (full[i]) gst_nt<u4>(A[i], val[i]);
#pragma unroll
        for (int i = 0; i < B; ++i)
            if (!full[i] && q0 + i * TC_PACK_THREADS < total) copy_partial<T>(v[i], A[i]);
    }
}

template <typename T, bool UNPACK>
hipError_t run(const PackKernelArgs& a, int K, int64_t nchunks, hipStream_t s) {
    dim3 grid(static_cast<unsigned>(nchunks), static_cast<unsigned>(K));
    hipLaunchKernelGGL((pack_kernel<T, UNPACK>), grid, dim3(TC_PACK_THREADS), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pack(const tc_tensorlist* tl, void* const* flat, bool unpack, bool /*flat_aligned*/,
                       hipStream_t stream) {
    const tc_group* g = tl->g;
    const tc_chunking& c = tl->elem == 2 ? g->sep2 : g->sep;
    PackKernelArgs a{};
    a.offsets = g->d_offsets;
    a.chunk_first = c.d_first;
    a.ptrs = tl->d_ptrs;
    a.n = g->n;
    a.N = g->N;
    a.chunk = c.chunk;
    for (int k = 0; k < tl->K; ++k) a.flat[k] = flat[k];
    if (tl->elem == 2)
        return unpack ? run<uint16_t, true>(a, tl->K, c.nchunks, stream)
                      : run<uint16_t, false>(a, tl->K, c.nchunks, stream);
    return unpack ? run<uint32_t, true>(a, tl->K, c.nchunks, stream)
                  : run<uint32_t, false>(a, tl->K, c.nchunks, stream);
}

}  // namespace tc
