// K-way reduction and fused elastic-averaging SGD step over flat copies.
//
// Both are streams over the flat index space with no reuse: every input is
// read once and every output written once, so they are bound by HBM
// bandwidth (well under one flop per byte) and use no matrix cores.
//
// Mapping: one lane owns one 16-byte slot of every stream (4 binary32
// values; 4 bfloat16 gradients are 8 bytes), so each wave instruction moves
// 1 KiB (512 B for bfloat16) of contiguous memory per buffer.  A lane issues
// the loads of all 2K+1 streams of its slot before any arithmetic, keeping
// (2K+1) x 16 B in flight per lane.  Workgroups walk the slots grid-stride.
// A ragged tail of fewer than 4 elements is handled element by element by
// the last workgroup; buffers that are not 16-byte aligned take the
// element-by-element kernel.
//
// The K terms are summed by a pairwise tree (adjacent pairs, level by level,
// an odd last term carried up) fully unrolled for K <= 16; larger K is
// summed as trees of 16 (zero-padded) combined by a tree of the partials.
#include "tc_internal.h"

#ifndef TC_EW_THREADS
#define TC_EW_THREADS 256
#endif
#ifndef TC_EW_BLOCKS_PER_CU
#define TC_EW_BLOCKS_PER_CU 8
#endif
#ifndef TC_NT_LOADS
#define TC_NT_LOADS 1
#endif
#ifndef TC_NT_STORES
#define TC_NT_STORES 1
#endif

namespace tc {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));

constexpr int kSpecialisedK = 16;

// ---------------------------------------------------------------- memory

template <typename T>
__device__ __forceinline__ T ld(const T* p) {
#if TC_NT_LOADS
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}

template <typename T>
__device__ __forceinline__ void st(T* p, T v) {
#if TC_NT_STORES
    __builtin_nontemporal_store(v, p);
#else
    *p = v;
#endif
}

// bfloat16 -> binary32 is exact: the bfloat16 code is the upper half of the
// binary32 code.
__device__ __forceinline__ float bf16_lo(unsigned int w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(unsigned int w) { return __uint_as_float(w & 0xffff0000u); }

// Value type V is f4 (one 16-byte slot, index = slot) or float (index =
// element).
template <typename V> struct Mem;

template <> struct Mem<f4> {
    static __device__ __forceinline__ f4 load(const float* p, int64_t i) {
        return ld(reinterpret_cast<const f4*>(p) + i);
    }
    static __device__ __forceinline__ f4 load(const uint16_t* p, int64_t i) {
        u2 w = ld(reinterpret_cast<const u2*>(p) + i);
        return f4{bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y)};
    }
    static __device__ __forceinline__ void store(float* p, int64_t i, f4 v) {
        st(reinterpret_cast<f4*>(p) + i, v);
    }
};

template <> struct Mem<float> {
    static __device__ __forceinline__ float load(const float* p, int64_t i) { return ld(p + i); }
    static __device__ __forceinline__ float load(const uint16_t* p, int64_t i) {
        return __uint_as_float(static_cast<unsigned int>(ld(p + i)) << 16);
    }
    static __device__ __forceinline__ void store(float* p, int64_t i, float v) { st(p + i, v); }
};

// ------------------------------------------------------------ arithmetic

__device__ __forceinline__ float fmav(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ __forceinline__ f4 fmav(f4 a, f4 b, f4 c) {
    return f4{__builtin_fmaf(a.x, b.x, c.x), __builtin_fmaf(a.y, b.y, c.y),
              __builtin_fmaf(a.z, b.z, c.z), __builtin_fmaf(a.w, b.w, c.w)};
}
template <typename V> __device__ __forceinline__ V splat(float s) { return V(s); }

// Pairwise tree over v[0..M): adjacent pairs level by level; an odd last
// element moves up unchanged.  Overwrites v.
template <int M> struct Tree {
    template <typename V> static __device__ __forceinline__ V sum(V* v) {
#pragma unroll
        for (int p = 0; p < M / 2; ++p) v[p] = v[2 * p] + v[2 * p + 1];
        if constexpr (M & 1) v[M / 2] = v[M - 1];
        return Tree<(M + 1) / 2>::sum(v);
    }
};
template <> struct Tree<1> {
    template <typename V> static __device__ __forceinline__ V sum(V* v) { return v[0]; }
};

// --------------------------------------------------------------- reduce

template <int K, typename T>
struct ReduceArgs {
    const T* in[K];
    float* out;
    int op;
    int k_total;  // the number of copies (== K except in the generic kernel)
};

template <int K, typename T, typename V>
__device__ __forceinline__ void reduce_slot(const ReduceArgs<K, T>& a, int64_t i) {
    V v[K];
#pragma unroll
    for (int q = 0; q < K; ++q) v[q] = Mem<V>::load(a.in[q], i);
    V s = Tree<K>::sum(v);
    if (a.op == TC_AVG) s = s / splat<V>(static_cast<float>(K));
    Mem<V>::store(a.out, i, s);
}

// Generic K (> kSpecialisedK): trees of 16 zero-padded, then a tree of the
// at most TC_MAX_K/16 partial sums (zero-padded).
template <typename T, typename V>
__device__ __forceinline__ void reduce_slot_generic(const ReduceArgs<TC_MAX_K, T>& a, int64_t i) {
    constexpr int kParts = TC_MAX_K / kSpecialisedK;
    V part[kParts];
#pragma unroll
    for (int c = 0; c < kParts; ++c) {
        V v[kSpecialisedK];
#pragma unroll
        for (int q = 0; q < kSpecialisedK; ++q) {
            const int k = c * kSpecialisedK + q;
            v[q] = k < a.k_total ? Mem<V>::load(a.in[k], i) : splat<V>(0.0f);
        }
        part[c] = Tree<kSpecialisedK>::sum(v);
    }
    V s = Tree<kParts>::sum(part);
    if (a.op == TC_AVG) s = s / splat<V>(static_cast<float>(a.k_total));
    Mem<V>::store(a.out, i, s);
}

template <int K, typename T>
__device__ __forceinline__ void reduce_any(const ReduceArgs<K, T>& a, int64_t i, f4) {
    if constexpr (K == TC_MAX_K) reduce_slot_generic<T, f4>(a, i); else reduce_slot<K, T, f4>(a, i);
}
template <int K, typename T>
__device__ __forceinline__ void reduce_any(const ReduceArgs<K, T>& a, int64_t i, float) {
    if constexpr (K == TC_MAX_K) reduce_slot_generic<T, float>(a, i); else reduce_slot<K, T, float>(a, i);
}

template <int K, typename T>
__global__ __launch_bounds__(TC_EW_THREADS) void reduce_vec_kernel(ReduceArgs<K, T> a, int64_t nslot, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * TC_EW_THREADS;
    for (int64_t s = static_cast<int64_t>(blockIdx.x) * TC_EW_THREADS + threadIdx.x; s < nslot; s += stride)
        reduce_any<K, T>(a, s, f4{});
    if (blockIdx.x == gridDim.x - 1) {
        const int64_t j = 4 * nslot + threadIdx.x;
        if (j < n) reduce_any<K, T>(a, j, 0.0f);
    }
}

template <int K, typename T>
__global__ __launch_bounds__(TC_EW_THREADS) void reduce_scalar_kernel(ReduceArgs<K, T> a, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * TC_EW_THREADS;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * TC_EW_THREADS + threadIdx.x; j < n; j += stride)
        reduce_any<K, T>(a, j, 0.0f);
}

// ---------------------------------------------------------------- easgd

template <int K, typename T>
struct EasgdArgs {
    float* x[K];
    const T* g[K];
    float* xc;
    float eta, rho, a;  // a = eta*rho rounded to binary32
    int k_total;
};

template <int K, typename T, typename V>
__device__ __forceinline__ void easgd_slot(const EasgdArgs<K, T>& a, int64_t i) {
    const V c = Mem<V>::load(a.xc, i);
    V x[K], g[K], d[K];
#pragma unroll
    for (int q = 0; q < K; ++q) {
        x[q] = Mem<V>::load(a.x[q], i);
        g[q] = Mem<V>::load(a.g[q], i);
    }
    const V rho = splat<V>(a.rho), neg_eta = splat<V>(-a.eta);
#pragma unroll
    for (int q = 0; q < K; ++q) {
        d[q] = x[q] - c;
        x[q] = fmav(neg_eta, fmav(rho, d[q], g[q]), x[q]);
    }
    const V cn = fmav(splat<V>(a.a), Tree<K>::sum(d), c);
#pragma unroll
    for (int q = 0; q < K; ++q) Mem<V>::store(a.x[q], i, x[q]);
    Mem<V>::store(a.xc, i, cn);
}

template <typename T, typename V>
__device__ __forceinline__ void easgd_slot_generic(const EasgdArgs<TC_MAX_K, T>& a, int64_t i) {
    constexpr int kParts = TC_MAX_K / kSpecialisedK;
    const V c = Mem<V>::load(a.xc, i);
    const V rho = splat<V>(a.rho), neg_eta = splat<V>(-a.eta);
    V part[kParts];
#pragma unroll
    for (int p = 0; p < kParts; ++p) {
        V d[kSpecialisedK];
#pragma unroll
        for (int q = 0; q < kSpecialisedK; ++q) {
            const int k = p * kSpecialisedK + q;
            if (k < a.k_total) {
                V x = Mem<V>::load(a.x[k], i);
                const V g = Mem<V>::load(a.g[k], i);
                d[q] = x - c;
                x = fmav(neg_eta, fmav(rho, d[q], g), x);
                Mem<V>::store(a.x[k], i, x);
            } else {
                d[q] = splat<V>(0.0f);
            }
        }
        part[p] = Tree<kSpecialisedK>::sum(d);
    }
    Mem<V>::store(a.xc, i, fmav(splat<V>(a.a), Tree<kParts>::sum(part), c));
}

template <int K, typename T>
__device__ __forceinline__ void easgd_any(const EasgdArgs<K, T>& a, int64_t i, f4) {
    if constexpr (K == TC_MAX_K) easgd_slot_generic<T, f4>(a, i); else easgd_slot<K, T, f4>(a, i);
}
template <int K, typename T>
__device__ __forceinline__ void easgd_any(const EasgdArgs<K, T>& a, int64_t i, float) {
    if constexpr (K == TC_MAX_K) easgd_slot_generic<T, float>(a, i); else easgd_slot<K, T, float>(a, i);
}

template <int K, typename T>
__global__ __launch_bounds__(TC_EW_THREADS) void easgd_vec_kernel(EasgdArgs<K, T> a, int64_t nslot, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * TC_EW_THREADS;
    for (int64_t s = static_cast<int64_t>(blockIdx.x) * TC_EW_THREADS + threadIdx.x; s < nslot; s += stride)
        easgd_any<K, T>(a, s, f4{});
    if (blockIdx.x == gridDim.x - 1) {
        const int64_t j = 4 * nslot + threadIdx.x;
        if (j < n) easgd_any<K, T>(a, j, 0.0f);
    }
}

template <int K, typename T>
__global__ __launch_bounds__(TC_EW_THREADS) void easgd_scalar_kernel(EasgdArgs<K, T> a, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * TC_EW_THREADS;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * TC_EW_THREADS + threadIdx.x; j < n; j += stride)
        easgd_any<K, T>(a, j, 0.0f);
}

// -------------------------------------------------------------- launching

int g_cu_count = 0;

int64_t grid_for(int64_t items) {
    if (g_cu_count == 0) {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
            g_cu_count = cus;
        else
            g_cu_count = 256;
    }
    const int64_t want = (items + TC_EW_THREADS - 1) / TC_EW_THREADS;
    const int64_t cap = static_cast<int64_t>(g_cu_count) * TC_EW_BLOCKS_PER_CU;
    return want < 1 ? 1 : (want < cap ? want : cap);
}

template <int K, typename T>
hipError_t run_reduce(const void* const* in, float* out, int op, int k_total, int64_t n, bool vec, hipStream_t s) {
    ReduceArgs<K, T> a{};
    for (int q = 0; q < k_total; ++q) a.in[q] = static_cast<const T*>(in[q]);
    a.out = out;
    a.op = op;
    a.k_total = k_total;
    if (vec) {
        const int64_t nslot = n / 4;
        hipLaunchKernelGGL((reduce_vec_kernel<K, T>), dim3(grid_for(nslot)), dim3(TC_EW_THREADS), 0, s, a, nslot, n);
    } else {
        hipLaunchKernelGGL((reduce_scalar_kernel<K, T>), dim3(grid_for(n)), dim3(TC_EW_THREADS), 0, s, a, n);
    }
    return hipGetLastError();
}

template <int K, typename T>
hipError_t run_easgd(float* const* x, const void* const* g, float* xc, float eta, float rho, int k_total,
                     int64_t n, bool vec, hipStream_t s) {
    EasgdArgs<K, T> a{};
    for (int q = 0; q < k_total; ++q) {
        a.x[q] = x[q];
        a.g[q] = static_cast<const T*>(g[q]);
    }
    a.xc = xc;
    a.eta = eta;
    a.rho = rho;
    a.a = eta * rho;  // one binary32 rounding, on the host
    a.k_total = k_total;
    if (vec) {
        const int64_t nslot = n / 4;
        hipLaunchKernelGGL((easgd_vec_kernel<K, T>), dim3(grid_for(nslot)), dim3(TC_EW_THREADS), 0, s, a, nslot, n);
    } else {
        hipLaunchKernelGGL((easgd_scalar_kernel<K, T>), dim3(grid_for(n)), dim3(TC_EW_THREADS), 0, s, a, n);
    }
    return hipGetLastError();
}

#define TC_FOR_K(X) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16)

template <typename T>
hipError_t dispatch_reduce(int K, const void* const* in, float* out, int op, int64_t n, bool vec, hipStream_t s) {
    switch (K) {
#define TC_CASE(k) \
    case k: return run_reduce<k, T>(in, out, op, K, n, vec, s);
        TC_FOR_K(TC_CASE)
#undef TC_CASE
        default: return run_reduce<TC_MAX_K, T>(in, out, op, K, n, vec, s);
    }
}

template <typename T>
hipError_t dispatch_easgd(int K, float* const* x, const void* const* g, float* xc, float eta, float rho, int64_t n,
                          bool vec, hipStream_t s) {
    switch (K) {
#define TC_CASE(k) \
    case k: return run_easgd<k, T>(x, g, xc, eta, rho, K, n, vec, s);
        TC_FOR_K(TC_CASE)
#undef TC_CASE
        default: return run_easgd<TC_MAX_K, T>(x, g, xc, eta, rho, K, n, vec, s);
    }
}

}  // namespace

hipError_t launch_reduce(int K, const void* const* in, int in_dtype, float* out, int op, int64_t n, bool vector_ok,
                         hipStream_t stream) {
    if (in_dtype == TC_BF16) return dispatch_reduce<uint16_t>(K, in, out, op, n, vector_ok, stream);
    return dispatch_reduce<float>(K, in, out, op, n, vector_ok, stream);
}

hipError_t launch_easgd(int K, float* const* x, const void* const* g, int g_dtype, float* xc, float eta, float rho,
                        int64_t n, bool vector_ok, hipStream_t stream) {
    if (g_dtype == TC_BF16) return dispatch_easgd<uint16_t>(K, x, g, xc, eta, rho, n, vector_ok, stream);
    return dispatch_easgd<float>(K, x, g, xc, eta, rho, n, vector_ok, stream);
}

}  // namespace tc
