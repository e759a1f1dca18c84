// Kernels on the tensor layout: the K copies of a group in one buffer,
// interleaved in slots of four elements (slot j of copy i at slot index
// j*K + i; Sec. 6.1 of the paper calls such a grouping of one vector per
// worker a "tensor").
//
// With the K copies interleaved, the fused step reads three streams (the
// workers, the gradients, the center) and writes two, instead of 2K+1 and
// K+1 separate buffers; the reduction reads one and writes one.  On MI355X
// this lifts the step from ~5.5 to ~6.4 TB/s: DRAM efficiency falls with
// the number of concurrent streams.
//
// Mapping: P = K rounded up to a power of two consecutive lanes own one
// slot, lane i holding worker i, so every wave instruction still moves 1 KiB
// of contiguous memory.  The K-way sums are cross-lane: quad permutes for
// partners l^1 and l^2, the half-row and row mirrors, then l^16 and l^32,
// which adds the terms in exactly the order of the pairwise tree the
// separate-buffer kernels use (lanes beyond K contribute 0).  The center is
// read by the P lanes of its slot (one coalesced access) and written by lane
// 0.  The last, partial slot of a group whose length is not a multiple of 4
// is done element by element by the last workgroup.
#include "tc_internal.h"

#ifndef TC_TP_BATCH
#define TC_TP_BATCH 2
#endif

namespace tc {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));

constexpr int next_pow2(int k) {
    int p = 1;
    while (p < k) p <<= 1;
    return p;
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    const int x = __builtin_bit_cast(int, v);
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(x, x, CTRL, 0xF, 0xF, false));
}

// Sum over each aligned group of P lanes; every lane of a group receives the
// group's sum (partners add the same two values, so all agree bit for bit).
template <int P>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr (P >= 2) v = v + dpp<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
    if constexpr (P >= 4) v = v + dpp<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
    if constexpr (P >= 8) v = v + dpp<0x141>(v);  // row_half_mirror: quad <-> quad
    if constexpr (P >= 16) v = v + dpp<0x140>(v); // row_mirror: half-row <-> half-row
    if constexpr (P >= 32) v = v + __shfl_xor(v, 16, 64);
    if constexpr (P >= 64) v = v + __shfl_xor(v, 32, 64);
    return v;
}

template <int P>
__device__ __forceinline__ f4 group_sum4(f4 v) {
    return f4{group_sum<P>(v.x), group_sum<P>(v.y), group_sum<P>(v.z), group_sum<P>(v.w)};
}

__device__ __forceinline__ f4 fma4(f4 a, f4 b, f4 c) {
    return f4{__builtin_fmaf(a.x, b.x, c.x), __builtin_fmaf(a.y, b.y, c.y), __builtin_fmaf(a.z, b.z, c.z),
              __builtin_fmaf(a.w, b.w, c.w)};
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// One slot (4 elements) of stored type T at slot index s of a buffer.
template <typename I>
__device__ __forceinline__ f4 load_slot(const float* p, I s) {
    return __builtin_nontemporal_load(reinterpret_cast<const f4*>(reinterpret_cast<const char*>(p) + s * I(16)));
}
template <typename I>
__device__ __forceinline__ f4 load_slot(const uint16_t* p, I s) {
    const u2 w = __builtin_nontemporal_load(reinterpret_cast<const u2*>(reinterpret_cast<const char*>(p) + s * I(8)));
    return f4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u), __uint_as_float(w.y << 16),
              __uint_as_float(w.y & 0xffff0000u)};
}
template <typename I>
__device__ __forceinline__ void store_slot(float* p, I s, f4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f4*>(reinterpret_cast<char*>(p) + s * I(16)));
}

__device__ __forceinline__ float load_elem(const float* p, int64_t e) { return p[e]; }
__device__ __forceinline__ float load_elem(const uint16_t* p, int64_t e) { return bf16_to_f32(p[e]); }

// Serial pairwise tree over P values (zero-padded beyond K), the order the
// lane butterfly uses; for the element-wise tail.
template <int M>
struct Tree {
    static __device__ __forceinline__ float sum(float* v) {
#pragma unroll
        for (int p = 0; p < M / 2; ++p) v[p] = v[2 * p] + v[2 * p + 1];
        return Tree<M / 2>::sum(v);
    }
};
template <>
struct Tree<1> {
    static __device__ __forceinline__ float sum(float* v) { return v[0]; }
};

// ------------------------------------------------------------- reduce

template <typename T>
struct TReduceArgs {
    const T* in;  // tensor layout, K copies
    float* out;   // N values
    int64_t nslot, n;
    int K, op;
};

// P: lanes per slot (K rounded up to a power of two).
template <int P, typename T, int U, typename I>
__global__ __launch_bounds__(256) void tensor_reduce_kernel(TReduceArgs<T> a) {
    constexpr int SPB = 256 / P;  // slots per workgroup and unroll step
    const int K = a.K;
    const int i = threadIdx.x % P;
    const I j0 = static_cast<I>(blockIdx.x) * SPB * U + threadIdx.x / P;
    const I nslot = static_cast<I>(a.nslot);
    f4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPB;
        v[u] = (j < nslot && i < K) ? load_slot(a.in, j * I(K) + I(i)) : f4(0.0f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPB;
        f4 s = group_sum4<P>(v[u]);
        if (a.op == TC_AVG) s = s / f4(static_cast<float>(K));  // correctly rounded
        if (j < nslot && i == 0) store_slot(a.out, j, s);
    }
    if (blockIdx.x == gridDim.x - 1) {  // trailing partial slot
        const int64_t e = 4 * a.nslot + threadIdx.x;
        if (e < a.n) {
            float t[P];
#pragma unroll
            for (int q = 0; q < P; ++q)
                t[q] = q < K ? load_elem(a.in, (a.nslot * K + q) * 4 + (e & 3)) : 0.0f;
            float s = Tree<P>::sum(t);
            if (a.op == TC_AVG) s = s / static_cast<float>(K);
            a.out[e] = s;
        }
    }
}

// --------------------------------------------------------------- easgd

template <typename T>
struct TEasgdArgs {
    float* x;        // tensor layout, K copies
    const T* g;      // tensor layout, K copies
    float* xc;       // N values
    int64_t nslot, n;
    float eta, rho, a;
    int K;
};

template <int P, typename T, int U, typename I>
__global__ __launch_bounds__(256) void tensor_easgd_kernel(TEasgdArgs<T> a) {
    constexpr int SPB = 256 / P;
    const int K = a.K;
    const int i = threadIdx.x % P;
    const I j0 = static_cast<I>(blockIdx.x) * SPB * U + threadIdx.x / P;
    const I nslot = static_cast<I>(a.nslot);
    f4 x[U], g[U], c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPB;
        const bool slot = j < nslot;
        c[u] = slot ? load_slot(a.xc, j) : f4(0.0f);
        const bool live = slot && i < K;
        x[u] = live ? load_slot(a.x, j * I(K) + I(i)) : f4(0.0f);
        g[u] = live ? load_slot(a.g, j * I(K) + I(i)) : f4(0.0f);
    }
    const f4 rho = f4(a.rho), neg_eta = f4(-a.eta), alpha = f4(a.a);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPB;
        const bool live = j < nslot && i < K;
        const f4 d = live ? x[u] - c[u] : f4(0.0f);
        const f4 xn = fma4(neg_eta, fma4(rho, d, g[u]), x[u]);
        const f4 cn = fma4(alpha, group_sum4<P>(d), c[u]);
        if (live) store_slot(a.x, j * I(K) + I(i), xn);
        if (j < nslot && i == 0) store_slot(a.xc, j, cn);
    }
    if (blockIdx.x == gridDim.x - 1) {  // trailing partial slot
        const int64_t e = 4 * a.nslot + threadIdx.x;
        if (e < a.n) {
            const float cv = a.xc[e];
            float d[P];
#pragma unroll
            for (int q = 0; q < P; ++q) {
                if (q < K) {
                    const int64_t idx = (a.nslot * K + q) * 4 + (e & 3);
                    const float xv = a.x[idx];
                    d[q] = xv - cv;
                    a.x[idx] = __builtin_fmaf(-a.eta, __builtin_fmaf(a.rho, d[q], load_elem(a.g, idx)), xv);
                } else {
                    d[q] = 0.0f;
                }
            }
            a.xc[e] = __builtin_fmaf(a.a, Tree<P>::sum(d), cv);
        }
    }
}

// ------------------------------------------------------- pack / unpack

struct TPackArgs {
    const int64_t* offsets;
    const int32_t* chunk_first;
    void* const* ptrs;  // K*n device pointers, copy-major
    void* tensor;       // tensor layout, K copies
    int32_t n, K;
    int64_t N, chunk;
};

__device__ __forceinline__ int32_t clamp_rel(int64_t v, int32_t clen) {
    return static_cast<int32_t>(v < 0 ? 0 : (v > clen ? clen : v));
}

// Bytes [sh, sh + 16) of the 32-byte little-endian concatenation lo:hi.
__device__ __forceinline__ u4 funnel(u4 lo, u4 hi, uint32_t sh) {
    const uint32_t w[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    const uint32_t d4 = sh >> 2, b = sh & 3;
    uint32_t t[5];
#pragma unroll
    for (int q = 0; q < 5; ++q)
        t[q] = d4 == 0 ? w[q] : d4 == 1 ? w[q + 1] : d4 == 2 ? w[q + 2] : w[q + 3];
    return u4{__builtin_amdgcn_alignbyte(t[1], t[0], b), __builtin_amdgcn_alignbyte(t[2], t[1], b),
              __builtin_amdgcn_alignbyte(t[3], t[2], b), __builtin_amdgcn_alignbyte(t[4], t[3], b)};
}

// SB source bytes at address S (SB = 16 or 8), read as the aligned 16-byte
// granule(s) holding them: only granules that contain some of the SB bytes
// are read.
template <int SB>
__device__ __forceinline__ u4 load_bytes(uintptr_t S) {
    if ((S & (SB - 1)) == 0) {
        if constexpr (SB == 16) return __builtin_nontemporal_load(reinterpret_cast<const u4*>(S));
        const u2 w = __builtin_nontemporal_load(reinterpret_cast<const u2*>(S));
        return u4{w.x, w.y, 0u, 0u};
    }
    const u4* g = reinterpret_cast<const u4*>(S & ~uintptr_t(15));
    const uint32_t sh = static_cast<uint32_t>(S & 15);
    const u4 g0 = g[0];
    const u4 g1 = sh + SB > 16 ? g[1] : g0;
    return funnel(g0, g1, sh);
}

template <int SB>
__device__ __forceinline__ void store_bytes(uintptr_t D, u4 v) {
    if constexpr (SB == 16) __builtin_nontemporal_store(v, reinterpret_cast<u4*>(D));
    else __builtin_nontemporal_store(u2{v.x, v.y}, reinterpret_cast<u2*>(D));
}

// Workgroup b moves chunk b of all K copies.  Pieces (slot, copy) are
// enumerated in tensor order, so the tensor side of every wave instruction
// is contiguous; the per-worker side reads or writes 4 elements of one
// copy's tensors, with one access when they lie in one tensor (funnel-
// shifted when misaligned on the read side), element by element otherwise.
template <typename T, bool UNPACK>
__global__ __launch_bounds__(256) void tensor_pack_kernel(TPackArgs a) {
    constexpr int ES = sizeof(T);
    constexpr int SB = 4 * ES;  // slot bytes
    constexpr int B = TC_TP_BATCH;
    __shared__ int32_t s_rel[kMaxStage + 1];
    __shared__ const char* s_ptr[kMaxStage];
    const int tid = threadIdx.x;
    const int64_t cstart = static_cast<int64_t>(blockIdx.x) * a.chunk;
    const int32_t clen = static_cast<int32_t>(a.N - cstart < a.chunk ? a.N - cstart : a.chunk);
    const int32_t lo = a.chunk_first[blockIdx.x];
    const int32_t hi = a.chunk_first[blockIdx.x + 1];
    const int nseg = hi - lo + 1;
    const int K = a.K;
    const int64_t first_start = a.offsets[lo] - cstart;
    const bool staged = static_cast<int64_t>(nseg) * K <= kMaxStage;  // pointers for all copies fit
    const bool rel_staged = nseg <= kMaxStage;
    for (int s = tid; s <= nseg && rel_staged; s += 256) s_rel[s] = clamp_rel(a.offsets[lo + s] - cstart, clen);
    if (staged)
        for (int q = tid; q < nseg * K; q += 256)
            s_ptr[q] = static_cast<const char*>(a.ptrs[static_cast<int64_t>(q / nseg) * a.n + lo + q % nseg]);
    __syncthreads();
    auto rel = [&](int s) -> int32_t {
        return rel_staged ? s_rel[s] : clamp_rel(a.offsets[lo + s] - cstart, clen);
    };
    auto ptr = [&](int k, int s) -> const char* {
        return staged ? s_ptr[k * nseg + s] : static_cast<const char*>(a.ptrs[static_cast<int64_t>(k) * a.n + lo + s]);
    };
    auto start = [&](int s) -> int64_t { return s == 0 ? first_start : rel(s); };
    auto find = [&](int jr) {  // last segment whose start is <= jr
        int l = 0, h = nseg - 1;
        while (l < h) {
            const int mid = (l + h + 1) >> 1;
            if (rel(mid) <= jr) l = mid; else h = mid - 1;
        }
        return l;
    };
    char* tens = static_cast<char*>(a.tensor);
    const int64_t slot0 = cstart / 4;
    const int nsl = clen / 4;  // whole slots in this chunk
    const int npieces = nsl * K;
    for (int q0 = tid; q0 < npieces; q0 += 256 * B) {
        u4 val[B];
        uintptr_t dst[B];
        bool vec[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int q = q0 + b * 256;
            vec[b] = false;
            if (q >= npieces) continue;
            const int js = q / K, k = q - js * K;
            const int jr = 4 * js;
            const uintptr_t piece = reinterpret_cast<uintptr_t>(tens) + ((slot0 + js) * K + k) * SB;
            int s = find(jr);
            if (jr + 4 <= rel(s + 1)) {
                const uintptr_t w = reinterpret_cast<uintptr_t>(ptr(k, s)) + (jr - start(s)) * ES;
                if (!UNPACK) {
                    val[b] = load_bytes<SB>(w);
                    dst[b] = piece;
                    vec[b] = true;
                } else if ((w & (SB - 1)) == 0) {
                    val[b] = load_bytes<SB>(piece);
                    dst[b] = w;
                    vec[b] = true;
                } else {
                    const T* src = reinterpret_cast<const T*>(piece);
                    T* d = reinterpret_cast<T*>(w);
#pragma unroll
                    for (int e = 0; e < 4; ++e) d[e] = src[e];
                }
            } else {  // the slot's 4 elements span tensors
                T* pc = reinterpret_cast<T*>(piece);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int je = jr + e;
                    while (je >= rel(s + 1)) ++s;
                    T* t = reinterpret_cast<T*>(const_cast<char*>(ptr(k, s))) + (je - start(s));
                    if (UNPACK) *t = pc[e];
                    else pc[e] = *t;
                }
            }
        }
#pragma unroll
        for (int b = 0; b < B; ++b)
            if (vec[b]) store_bytes<SB>(dst[b], val[b]);
    }
    // the group's last, partial slot: element by element, every copy
    const int rem = clen - 4 * nsl;
    if (tid < rem * K) {
        const int k = tid / rem, e = tid - k * rem;
        const int je = 4 * nsl + e;
        int s = find(je);
        while (je >= rel(s + 1)) ++s;
        T* t = reinterpret_cast<T*>(const_cast<char*>(ptr(k, s))) + (je - start(s));
        T* pc = reinterpret_cast<T*>(tens) + ((slot0 + nsl) * K + k) * 4 + e;
        if (UNPACK) *t = *pc;
        else *pc = *t;
    }
}

// ---------------------------------------------------------- launching

// Slots per lane: two for the reduction, one for the step (measured).
constexpr int kTReduceUnroll = 2;
constexpr int kTEasgdUnroll = 1;

template <int P, typename T>
hipError_t run_treduce(int K, const void* in, float* out, int op, int64_t n, hipStream_t s) {
    constexpr int U = kTReduceUnroll;
    constexpr int SPB = 256 / P;
    TReduceArgs<T> a{static_cast<const T*>(in), out, n / 4, n, K, op};
    const int64_t blocks = (a.nslot + SPB * U - 1) / (SPB * U);
    dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
    if ((a.nslot + 1) * K * 16 < (int64_t(1) << 32))
        hipLaunchKernelGGL((tensor_reduce_kernel<P, T, U, uint32_t>), grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((tensor_reduce_kernel<P, T, U, int64_t>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int P, typename T>
hipError_t run_teasgd(int K, float* x, const void* g, float* xc, float eta, float rho, int64_t n, hipStream_t s) {
    constexpr int U = kTEasgdUnroll;
    constexpr int SPB = 256 / P;
    TEasgdArgs<T> a{x, static_cast<const T*>(g), xc, n / 4, n, eta, rho, eta * rho, K};
    const int64_t blocks = (a.nslot + SPB * U - 1) / (SPB * U);
    dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
    if ((a.nslot + 1) * K * 16 < (int64_t(1) << 32))
        hipLaunchKernelGGL((tensor_easgd_kernel<P, T, U, uint32_t>), grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((tensor_easgd_kernel<P, T, U, int64_t>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

#define TC_FOR_P(X) X(1) X(2) X(4) X(8) X(16) X(32) X(64)

template <typename T>
hipError_t dispatch_treduce(int K, const void* in, float* out, int op, int64_t n, hipStream_t s) {
    switch (next_pow2(K)) {
#define TC_CASE(p) \
    case p: return run_treduce<p, T>(K, in, out, op, n, s);
        TC_FOR_P(TC_CASE)
#undef TC_CASE
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t dispatch_teasgd(int K, float* x, const void* g, float* xc, float eta, float rho, int64_t n,
                           hipStream_t s) {
    switch (next_pow2(K)) {
#define TC_CASE(p) \
    case p: return run_teasgd<p, T>(K, x, g, xc, eta, rho, n, s);
        TC_FOR_P(TC_CASE)
#undef TC_CASE
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_tensor_reduce(int K, const void* in, int in_dtype, float* out, int op, int64_t n,
                                hipStream_t stream) {
    if (in_dtype == TC_BF16) return dispatch_treduce<uint16_t>(K, in, out, op, n, stream);
    return dispatch_treduce<float>(K, in, out, op, n, stream);
}

hipError_t launch_tensor_easgd(int K, float* x, const void* g, int g_dtype, float* xc, float eta, float rho,
                               int64_t n, hipStream_t stream) {
    if (g_dtype == TC_BF16) return dispatch_teasgd<uint16_t>(K, x, g, xc, eta, rho, n, stream);
    return dispatch_teasgd<float>(K, x, g, xc, eta, rho, n, stream);
}

hipError_t launch_tensor_pack(const tc_tensorlist* tl, void* tensor, bool unpack, hipStream_t stream) {
    const tc_group* g = tl->g;
    TPackArgs a{g->d_offsets, g->d_chunk_first, tl->d_ptrs, tensor, g->n, tl->K, g->N, g->chunk};
    dim3 grid(static_cast<unsigned>(g->nchunks));
    if (tl->elem == 2) {
        if (unpack) hipLaunchKernelGGL((tensor_pack_kernel<uint16_t, true>), grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((tensor_pack_kernel<uint16_t, false>), grid, dim3(256), 0, stream, a);
    } else {
        if (unpack) hipLaunchKernelGGL((tensor_pack_kernel<uint32_t, true>), grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((tensor_pack_kernel<uint32_t, false>), grid, dim3(256), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace tc
