// K-way reduction and fused elastic-averaging SGD step over flat copies.
//
// Both are streams over the flat index space with no reuse: every input is
// read once and every output written once, so they are bound by HBM
// bandwidth (well under one flop per byte) and use no matrix cores.
//
// Mapping: one lane owns one 16-byte slot of every stream (4 binary32
// values; 4 bfloat16 gradients are 8 bytes), so each wave instruction moves
// 1 KiB (512 B for bfloat16) of contiguous memory per buffer.  A lane owns
// U slots (U = 4, 2 or 1 as K grows) and issues the loads of all streams of
// all of them before any arithmetic.  One workgroup per tile of 256*U
// slots; non-temporal loads and stores, since nothing is re-read.
// A ragged tail of fewer than 4 elements is handled element by element by
// the last workgroup; buffers that are not 16-byte aligned take the
// element-by-element kernel.
//
// The K terms are summed by a pairwise tree (adjacent pairs, level by level,
// an odd last term carried up) fully unrolled for K <= 16; larger K is
// summed as trees of 16 (zero-padded) combined by a tree of the four
// partials (zero-padded).  The kernels for K > 16 loop over the groups of 16
// copies without unrolling, so that only one group's pointers are live: fully
// unrolled over 64 copies they held 128 pointer SGPRs, spilled 120-770 SGPRs
// into VGPR lanes and ran at one wave per SIMD (measured on MI355X, ResNet-50
// group at K = 32: bfloat16 reduction 1.07 TB/s, binary32 fused step 3.9).
#include "tc_internal.h"

#ifndef TC_EW_THREADS
#define TC_EW_THREADS 256
#endif
// Workgroups per CU when the grid is capped; 0 launches one workgroup per
// tile of TC_EW_THREADS * unroll slots (measured fastest on MI355X: the
// dispatcher then keeps the active window of every stream compact).
#ifndef TC_EW_BLOCKS_PER_CU
#define TC_EW_BLOCKS_PER_CU 0
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
typedef unsigned int u4 __attribute__((ext_vector_type(4)));

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

// Value type V is f4 (one 16-byte slot; index = slot) or float (index =
// element).  Index type I is uint32_t when every buffer is below 4 GiB: the
// address is then a uniform 64-bit base plus one 32-bit byte offset that all
// streams share, which the compiler emits as SGPR-base + VGPR-offset loads
// and stores instead of one 64-bit VGPR address per stream.
template <typename I>
__device__ __forceinline__ const char* at(const void* p, I byte_off) {
    return static_cast<const char*>(p) + byte_off;
}

template <typename V> struct Mem;

template <> struct Mem<f4> {
    template <typename I> static __device__ __forceinline__ f4 load(const float* p, I i) {
        return ld(reinterpret_cast<const f4*>(at(p, i * I(16))));
    }
    template <typename I> static __device__ __forceinline__ f4 load(const uint16_t* p, I i) {
        u2 w = ld(reinterpret_cast<const u2*>(at(p, i * I(8))));
        return f4{bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y)};
    }
    template <typename I> static __device__ __forceinline__ void store(float* p, I i, f4 v) {
        st(reinterpret_cast<f4*>(const_cast<char*>(at(p, i * I(16)))), v);
    }
};

template <> struct Mem<float> {
    template <typename I> static __device__ __forceinline__ float load(const float* p, I i) {
        return ld(reinterpret_cast<const float*>(at(p, i * I(4))));
    }
    template <typename I> static __device__ __forceinline__ float load(const uint16_t* p, I i) {
        return __uint_as_float(static_cast<unsigned int>(ld(reinterpret_cast<const uint16_t*>(at(p, i * I(2))))) << 16);
    }
    template <typename I> static __device__ __forceinline__ void store(float* p, I i, float v) {
        st(reinterpret_cast<float*>(const_cast<char*>(at(p, i * I(4)))), v);
    }
};

// Output stores with explicit cache-policy bits (bit 0 sc0, bit 1 nt, bit 4
// sc1), as raw buffer stores when offsets are 32-bit; a negative policy
// keeps the plain non-temporal global store.  Measured on MI355X: the
// reduction's single output stream is 4-6% faster with sc1 than with nt.
#ifndef TC_RD_STORE_AUX
#define TC_RD_STORE_AUX 16
#endif
#ifndef TC_EA_X_STORE_AUX
#define TC_EA_X_STORE_AUX -1
#endif
#ifndef TC_EA_C_STORE_AUX
#define TC_EA_C_STORE_AUX -1
#endif

template <int AUX, typename V, typename I>
__device__ __forceinline__ void store_pol(float* p, I i, V v, uint32_t bytes) {
    if constexpr (AUX >= 0 && sizeof(I) == 4 && sizeof(V) == 16) {
        const __amdgpu_buffer_rsrc_t r =
            __builtin_amdgcn_make_buffer_rsrc(p, static_cast<short>(0), static_cast<int>(bytes), 0x00020000);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), r, i * 16u, 0, AUX);
    } else {
        Mem<V>::store(p, i, v);
    }
}

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
    uint32_t out_bytes;  // size of out when below 4 GiB
    int op;
    int k_total;  // the number of copies (== K except in the generic kernel)
};

// U slots per lane at a time (slot i + u*TC_EW_THREADS), all loads first.
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void reduce_slots(const ReduceArgs<K, T>& a, I i, I du) {
    V v[U][K];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int q = 0; q < K; ++q) v[u][q] = Mem<V>::load(a.in[q], i + I(u) * du);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        V s = Tree<K>::sum(v[u]);
        if (a.op == TC_AVG) s = s / splat<V>(static_cast<float>(K));
        store_pol<TC_RD_STORE_AUX, V, I>(a.out, i + I(u) * du, s, a.out_bytes);
    }
}

// Generic K (> kSpecialisedK): the partial sums of the groups of 16 copies
// (each a tree of 16, zero-padded) kept in four registers, +0 for a group
// past k_total, and combined as the tree of four: (p0 + p1) + (p2 + p3).
static_assert(TC_MAX_K == 4 * kSpecialisedK, "the generic kernels combine four groups of 16 copies");

template <typename V>
struct Parts {
    V p0 = splat<V>(0.0f), p1 = splat<V>(0.0f), p2 = splat<V>(0.0f), p3 = splat<V>(0.0f);
    __device__ __forceinline__ void set(int c, V p) {
        p0 = c == 0 ? p : p0;
        p1 = c == 1 ? p : p1;
        p2 = c == 2 ? p : p2;
        p3 = c == 3 ? p : p3;
    }
    __device__ __forceinline__ V sum() const { return (p0 + p1) + (p2 + p3); }
};

// Every load of a group before its sums.  A full group of 16 copies loads
// without conditions: a load under a condition compiled, for bfloat16
// inputs, to a branch around it and a wait for it, one load in flight at a
// time (measured on MI355X, ResNet-50 group: K = 17-64 4.1-4.2 TB/s, against
// 5.8-6.2 without the conditions); a last, partial group keeps them and
// loads only its copies (K = 17 in binary32: 9% faster than loading 16).
template <typename T, typename V, typename I>
__device__ __forceinline__ void reduce_slot_generic(const ReduceArgs<TC_MAX_K, T>& a, I i) {
    Parts<V> parts;
    const int groups = (a.k_total + kSpecialisedK - 1) / kSpecialisedK;
#pragma unroll 1
    for (int c = 0; c < groups; ++c) {
        V v[kSpecialisedK];
        if ((c + 1) * kSpecialisedK <= a.k_total) {
#pragma unroll
            for (int q = 0; q < kSpecialisedK; ++q) v[q] = Mem<V>::load(a.in[c * kSpecialisedK + q], i);
        } else {
#pragma unroll
            for (int q = 0; q < kSpecialisedK; ++q) {
                const int k = c * kSpecialisedK + q;
                v[q] = k < a.k_total ? Mem<V>::load(a.in[k], i) : splat<V>(0.0f);
            }
        }
        parts.set(c, Tree<kSpecialisedK>::sum(v));
    }
    V s = parts.sum();
    if (a.op == TC_AVG) s = s / splat<V>(static_cast<float>(a.k_total));
    Mem<V>::store(a.out, i, s);
}

template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void reduce_any(const ReduceArgs<K, T>& a, I i, I du) {
    if constexpr (K == TC_MAX_K) reduce_slot_generic<T, V, I>(a, i);
    else reduce_slots<K, T, U, V, I>(a, i, du);
}

// ---------------------------------------------------------------- easgd

template <int K, typename T>
struct EasgdArgs {
    float* x[K];
    const T* g[K];
    float* xc;
    uint32_t bytes;     // size of each x buffer and of xc when below 4 GiB
    float eta, rho, a;  // a = eta*rho rounded to binary32
    int k_total;
    static constexpr bool kReduce = false;
};

// The step fused with the K-way reduction of the gradients it reads: out =
// the SUM (or AVG) of g_0 .. g_{K-1}, by the reduction's own tree and
// quotient, so the result is bit for bit that of the reduction call.
template <int K, typename T>
struct ReduceEasgdArgs : EasgdArgs<K, T> {
    float* out;
    int op;
    static constexpr bool kReduce = true;
};

template <int K, typename T, int U, typename V, typename I, typename A>
__device__ __forceinline__ void easgd_slots(const A& a, I i, I du) {
    V c[U], x[U][K], g[U][K], r[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        c[u] = Mem<V>::load(a.xc, i + I(u) * du);
#pragma unroll
        for (int q = 0; q < K; ++q) {
            x[u][q] = Mem<V>::load(a.x[q], i + I(u) * du);
            g[u][q] = Mem<V>::load(a.g[q], i + I(u) * du);
        }
    }
    const V rho = splat<V>(a.rho), neg_eta = splat<V>(-a.eta), alpha = splat<V>(a.a);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        V d[K];
#pragma unroll
        for (int q = 0; q < K; ++q) {
            d[q] = x[u][q] - c[u];
            x[u][q] = fmav(neg_eta, fmav(rho, d[q], g[u][q]), x[u][q]);
        }
        c[u] = fmav(alpha, Tree<K>::sum(d), c[u]);
        if constexpr (A::kReduce) {
            r[u] = Tree<K>::sum(g[u]);
            if (a.op == TC_AVG) r[u] = r[u] / splat<V>(static_cast<float>(K));
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int q = 0; q < K; ++q) store_pol<TC_EA_X_STORE_AUX, V, I>(a.x[q], i + I(u) * du, x[u][q], a.bytes);
        store_pol<TC_EA_C_STORE_AUX, V, I>(a.xc, i + I(u) * du, c[u], a.bytes);
        if constexpr (A::kReduce) store_pol<TC_RD_STORE_AUX, V, I>(a.out, i + I(u) * du, r[u], a.bytes);
    }
}

// Generic K: per group of 16 workers, every load before the first store (a
// store to one worker's buffer would otherwise order the next worker's loads
// behind it).
template <typename T, typename V, typename I, typename A>
__device__ __forceinline__ void easgd_slot_generic(const A& a, I i) {
    const V c = Mem<V>::load(a.xc, i);
    const V rho = splat<V>(a.rho), neg_eta = splat<V>(-a.eta);
    Parts<V> parts, gparts;
    const int groups = (a.k_total + kSpecialisedK - 1) / kSpecialisedK;
#pragma unroll 1
    for (int p = 0; p < groups; ++p) {
        V x[kSpecialisedK], g[kSpecialisedK], d[kSpecialisedK];
#pragma unroll
        for (int q = 0; q < kSpecialisedK; ++q) {
            const int k = p * kSpecialisedK + q;
            x[q] = k < a.k_total ? Mem<V>::load(a.x[k], i) : splat<V>(0.0f);
            g[q] = k < a.k_total ? Mem<V>::load(a.g[k], i) : splat<V>(0.0f);
        }
#pragma unroll
        for (int q = 0; q < kSpecialisedK; ++q) {
            d[q] = p * kSpecialisedK + q < a.k_total ? x[q] - c : splat<V>(0.0f);  // +0 past k_total
            x[q] = fmav(neg_eta, fmav(rho, d[q], g[q]), x[q]);
        }
#pragma unroll
        for (int q = 0; q < kSpecialisedK; ++q)
            if (p * kSpecialisedK + q < a.k_total) Mem<V>::store(a.x[p * kSpecialisedK + q], i, x[q]);
        parts.set(p, Tree<kSpecialisedK>::sum(d));
        // the gradients past k_total are +0, as in the reduction's last group
        if constexpr (A::kReduce) gparts.set(p, Tree<kSpecialisedK>::sum(g));
    }
    Mem<V>::store(a.xc, i, fmav(splat<V>(a.a), parts.sum(), c));
    if constexpr (A::kReduce) {
        V s = gparts.sum();
        if (a.op == TC_AVG) s = s / splat<V>(static_cast<float>(a.k_total));
        Mem<V>::store(a.out, i, s);
    }
}

template <int K, typename T, int U, typename V, typename I, typename A>
__device__ __forceinline__ void easgd_any(const A& a, I i, I du) {
    if constexpr (K == TC_MAX_K) easgd_slot_generic<T, V, I>(a, i);
    else easgd_slots<K, T, U, V, I>(a, i, du);
}

// ---------------------------------------------------- sgd / sync / async

// Plain SGD on every worker: x_i = fma(-eta, g_i, x_i).
template <int K, typename T>
struct SgdArgs {
    float* x[K];
    const T* g[K];
    float eta;
    int k_total;
};

template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void sgd_slots(const SgdArgs<K, T>& a, I i, I du) {
    if constexpr (K == TC_MAX_K) {
        for (int q = 0; q < a.k_total; ++q) {  // workers one at a time
            const V x = Mem<V>::load(a.x[q], i), g = Mem<V>::load(a.g[q], i);
            Mem<V>::store(a.x[q], i, fmav(splat<V>(-a.eta), g, x));
        }
    } else {
        V x[U][K], g[U][K];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int q = 0; q < K; ++q) {
                x[u][q] = Mem<V>::load(a.x[q], i + I(u) * du);
                g[u][q] = Mem<V>::load(a.g[q], i + I(u) * du);
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int q = 0; q < K; ++q) Mem<V>::store(a.x[q], i + I(u) * du, fmav(splat<V>(-a.eta), g[u][q], x[u][q]));
    }
}

// Synchronous SGD through pushpull: S = pairwise sum of the K gradients,
// x_i = fma(-eta*rescale, S, x_i) for every worker, and, when broadcast,
// g_i = S (binary32 gradients only).
template <int K, typename T>
struct SyncArgs {
    float* x[K];
    T* g[K];
    float step;  // eta * rescale, rounded once to binary32
    int broadcast;
    int k_total;
};

template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void sync_slots(const SyncArgs<K, T>& a, I i, I du) {
    if constexpr (K == TC_MAX_K) {
        Parts<V> parts;
        const int groups = (a.k_total + kSpecialisedK - 1) / kSpecialisedK;
#pragma unroll 1
        for (int c = 0; c < groups; ++c) {
            V v[kSpecialisedK];
#pragma unroll
            for (int q = 0; q < kSpecialisedK; ++q) {
                const int k = c * kSpecialisedK + q;
                v[q] = k < a.k_total ? Mem<V>::load(static_cast<const T*>(a.g[k]), i) : splat<V>(0.0f);
            }
            parts.set(c, Tree<kSpecialisedK>::sum(v));
        }
        const V S = parts.sum();
        // the workers in groups of 16, every load before the first store
#pragma unroll 1
        for (int c = 0; c < groups; ++c) {
            V x[kSpecialisedK];
#pragma unroll
            for (int q = 0; q < kSpecialisedK; ++q) {
                const int k = c * kSpecialisedK + q;
                if (k < a.k_total) x[q] = Mem<V>::load(a.x[k], i);
            }
#pragma unroll
            for (int q = 0; q < kSpecialisedK; ++q) {
                const int k = c * kSpecialisedK + q;
                if (k < a.k_total) {
                    Mem<V>::store(a.x[k], i, fmav(splat<V>(-a.step), S, x[q]));
                    if constexpr (sizeof(T) == 4)
                        if (a.broadcast) Mem<V>::store(a.g[k], i, S);
                }
            }
        }
    } else {
        V g[U][K], x[U][K];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int q = 0; q < K; ++q) {
                g[u][q] = Mem<V>::load(static_cast<const T*>(a.g[q]), i + I(u) * du);
                x[u][q] = Mem<V>::load(a.x[q], i + I(u) * du);
            }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const V S = Tree<K>::sum(g[u]);
#pragma unroll
            for (int q = 0; q < K; ++q) {
                Mem<V>::store(a.x[q], i + I(u) * du, fmav(splat<V>(-a.step), S, x[u][q]));
                if constexpr (sizeof(T) == 4)
                    if (a.broadcast) Mem<V>::store(a.g[q], i + I(u) * du, S);
            }
        }
    }
}

// Asynchronous elastic exchanges: for r < R, worker w = order[r] (no worker
// twice): d = x_w - c; c = fma(alpha, d, c); x_w = fma(-alpha, d, x_w).
constexpr int kMaxOrder = TC_MAX_K;
template <int K>
struct AsyncArgs {
    float* x[K];
    float* xc;
    uint8_t order[kMaxOrder];
    int R;
    float alpha;
    int k_total;
};

template <int K, typename T>
struct AsyncArgsT : AsyncArgs<K> {};

template <int K, int U, typename V, typename I>
__device__ __forceinline__ void async_slots(const AsyncArgs<K>& a, I i, I du) {
    if constexpr (K == TC_MAX_K) {
        V c = Mem<V>::load(a.xc, i);
        for (int r = 0; r < a.R; ++r) {  // exchanges one at a time
            float* xw = a.x[a.order[r]];
            V x = Mem<V>::load(xw, i);
            const V d = x - c;
            c = fmav(splat<V>(a.alpha), d, c);
            Mem<V>::store(xw, i, fmav(splat<V>(-a.alpha), d, x));
        }
        Mem<V>::store(a.xc, i, c);
    } else {
        // the (distinct) exchanged workers' values are all loaded first
        V c[U], x[U][K];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            c[u] = Mem<V>::load(a.xc, i + I(u) * du);
#pragma unroll
            for (int r = 0; r < K; ++r)
                if (r < a.R) x[u][r] = Mem<V>::load(a.x[a.order[r]], i + I(u) * du);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int r = 0; r < K; ++r)
                if (r < a.R) {
                    const V d = x[u][r] - c[u];
                    c[u] = fmav(splat<V>(a.alpha), d, c[u]);
                    x[u][r] = fmav(splat<V>(-a.alpha), d, x[u][r]);
                }
#pragma unroll
            for (int r = 0; r < K; ++r)
                if (r < a.R) Mem<V>::store(a.x[a.order[r]], i + I(u) * du, x[u][r]);
            Mem<V>::store(a.xc, i + I(u) * du, c[u]);
        }
    }
}

// -------------------------------------------------------------- kernels

// The operation is selected by the argument type.
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void op_any(const ReduceArgs<K, T>& a, I i, I du) { reduce_any<K, T, U, V, I>(a, i, du); }
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void op_any(const EasgdArgs<K, T>& a, I i, I du) { easgd_any<K, T, U, V, I>(a, i, du); }
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void op_any(const ReduceEasgdArgs<K, T>& a, I i, I du) {
    easgd_any<K, T, U, V, I>(a, i, du);
}
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void op_any(const SgdArgs<K, T>& a, I i, I du) { sgd_slots<K, T, U, V, I>(a, i, du); }
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void op_any(const SyncArgs<K, T>& a, I i, I du) { sync_slots<K, T, U, V, I>(a, i, du); }
template <int K, typename T, int U, typename V, typename I>
__device__ __forceinline__ void op_any(const AsyncArgsT<K, T>& a, I i, I du) { async_slots<K, U, V, I>(a, i, du); }
// 16-byte slots, grid-stride; groups of U slots per lane, then the slots of
// a last partial group one by one; the last workgroup does the < 4
// trailing elements.
template <int K, typename T, int U, typename I, template <int, typename> class Args>
__global__ __launch_bounds__(TC_EW_THREADS) void vec_kernel(Args<K, T> a, I nslot, I n) {
    constexpr int kU = (K == TC_MAX_K) ? 1 : U;
    const I T_ = TC_EW_THREADS;
    const I stride = static_cast<I>(gridDim.x) * T_ * kU;
    I s = static_cast<I>(blockIdx.x) * T_ * kU + threadIdx.x;
    for (; s + I(kU - 1) * T_ < nslot; s += stride) op_any<K, T, kU, f4, I>(a, s, T_);
#pragma unroll
    for (int u = 0; u < kU - 1; ++u)
        if (s + I(u) * T_ < nslot) op_any<K, T, 1, f4, I>(a, s + I(u) * T_, T_);
    if (blockIdx.x == gridDim.x - 1) {
        const I j = 4 * nslot + threadIdx.x;
        if (j < n) op_any<K, T, 1, float, I>(a, j, I(1));
    }
}

// Element by element, grid-stride (buffers not 16-byte aligned).
template <int K, typename T, typename I, template <int, typename> class Args>
__global__ __launch_bounds__(TC_EW_THREADS) void scalar_kernel(Args<K, T> a, I n) {
    const I stride = static_cast<I>(gridDim.x) * TC_EW_THREADS;
    for (I j = static_cast<I>(blockIdx.x) * TC_EW_THREADS + threadIdx.x; j < n; j += stride)
        op_any<K, T, 1, float, I>(a, j, I(1));
}

// -------------------------------------------------------------- launching

// Slots per lane in flight, by the number of streams: more slots for few
// streams, one slot once a lane already has 2K+1 >= 17 loads in flight
// (measured on MI355X; more costs occupancy without adding bandwidth).
constexpr int reduce_unroll(int K) { return K <= 3 ? 4 : K <= 8 ? 2 : 1; }
// bfloat16 inputs load 8-byte slots: twice the slots keep as many bytes in
// flight (measured at K = 16: 6.26 -> 6.35-6.41 TB/s; four times: 4.3)
constexpr int kBf16ReduceScale = 2;
constexpr int easgd_unroll(int K) { return K <= 2 ? 4 : K <= 8 ? 2 : 1; }

int g_cu_count = 0;

int64_t grid_for(int64_t items, int per_lane) {
    if (g_cu_count == 0) {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
            g_cu_count = cus;
        else
            g_cu_count = 256;
    }
    const int64_t per_block = static_cast<int64_t>(TC_EW_THREADS) * per_lane;
    const int64_t want = (items + per_block - 1) / per_block;
    if (TC_EW_BLOCKS_PER_CU <= 0) return want < 1 ? 1 : want;
    const int64_t cap = static_cast<int64_t>(g_cu_count) * TC_EW_BLOCKS_PER_CU;
    return want < 1 ? 1 : (want < cap ? want : cap);
}

template <int K, typename T, int U, template <int, typename> class Args>
hipError_t launch(const Args<K, T>& a, int64_t n, bool vec, int elem_bytes_max, hipStream_t s) {
    // 32-bit byte offsets when the largest buffer is below 4 GiB
    const bool off32 = n * elem_bytes_max < (int64_t(1) << 32) - 64;
    if (vec) {
        const int64_t nslot = n / 4;
        dim3 grid(static_cast<unsigned>(grid_for(nslot, K == TC_MAX_K ? 1 : U)));
        if (off32)
            hipLaunchKernelGGL((vec_kernel<K, T, U, uint32_t, Args>), grid, dim3(TC_EW_THREADS), 0, s, a,
                               static_cast<uint32_t>(nslot), static_cast<uint32_t>(n));
        else
            hipLaunchKernelGGL((vec_kernel<K, T, U, int64_t, Args>), grid, dim3(TC_EW_THREADS), 0, s, a, nslot, n);
    } else {
        dim3 grid(static_cast<unsigned>(grid_for(n, 1)));
        if (off32)
            hipLaunchKernelGGL((scalar_kernel<K, T, uint32_t, Args>), grid, dim3(TC_EW_THREADS), 0, s, a,
                               static_cast<uint32_t>(n));
        else
            hipLaunchKernelGGL((scalar_kernel<K, T, int64_t, Args>), grid, dim3(TC_EW_THREADS), 0, s, a, n);
    }
    return hipGetLastError();
}

template <int K, typename T>
hipError_t run_reduce(const void* const* in, float* out, int op, int k_total, int64_t n, bool vec, hipStream_t s) {
    ReduceArgs<K, T> a{};
    for (int q = 0; q < k_total; ++q) a.in[q] = static_cast<const T*>(in[q]);
    a.out = out;
    a.out_bytes = n * 4 < (int64_t(1) << 32) ? static_cast<uint32_t>(n * 4) : 0;
    a.op = op;
    a.k_total = k_total;
    return launch<K, T, reduce_unroll(K) * (sizeof(T) == 2 ? kBf16ReduceScale : 1)>(a, n, vec, 4, s);
}

template <int K, typename T>
hipError_t run_easgd(float* const* x, const void* const* g, float* xc, float* out, int op, float eta, float rho,
                     int k_total, int64_t n, bool vec, hipStream_t s) {
    ReduceEasgdArgs<K, T> a{};
    for (int q = 0; q < k_total; ++q) {
        a.x[q] = x[q];
        a.g[q] = static_cast<const T*>(g[q]);
    }
    a.xc = xc;
    a.bytes = n * 4 < (int64_t(1) << 32) ? static_cast<uint32_t>(n * 4) : 0;
    a.eta = eta;
    a.rho = rho;
    a.a = eta * rho;  // one binary32 rounding, on the host
    a.k_total = k_total;
    a.out = out;
    a.op = op;
    if (out) return launch<K, T, easgd_unroll(K)>(a, n, vec, 4, s);
    return launch<K, T, easgd_unroll(K)>(static_cast<const EasgdArgs<K, T>&>(a), n, vec, 4, s);
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
hipError_t dispatch_easgd(int K, float* const* x, const void* const* g, float* xc, float* out, int op, float eta,
                          float rho, int64_t n, bool vec, hipStream_t s) {
    switch (K) {
#define TC_CASE(k) \
    case k: return run_easgd<k, T>(x, g, xc, out, op, eta, rho, K, n, vec, s);
        TC_FOR_K(TC_CASE)
#undef TC_CASE
        default: return run_easgd<TC_MAX_K, T>(x, g, xc, out, op, eta, rho, K, n, vec, s);
    }
}

// Broadcast of one flat buffer to K copies, bit for bit: 16-byte slots when
// every buffer is 16-byte aligned, element by element otherwise; the last
// workgroup copies the bytes after the last whole slot.
//
// Slot path: a workgroup copies one chunk of TC_EW_THREADS slots of the
// source into C of the copies.  The grid runs window by window (window
// chunks of the source each): within a window, the chunks for copies 0..C-1
// come first, then those for copies C..2C-1, and so on, so that the
// workgroups resident at one time write about C copies rather than all K,
// and the later passes over a window find its source in the last-level
// cache.  The source is read with ordinary (cacheable) loads for that reuse.
// Measured on MI355X with calls rotating over sources that total > 768 MB,
// so no call finds its source cached by an earlier one (GB/s; ResNet-50
// group K = 8 / 16 / 4, VGG-16 group K = 8 / 4): every copy per workgroup
// with non-temporal source loads 4,458-4,490 / 4,912-4,931 / 5,094-5,145 /
// 5,155-5,200 / 5,198-5,270; C = 4 over windows of 8,192 chunks (32 MiB of
// binary32 source) 5,297-5,329 / 5,295-5,337 / 5,325-5,354 / 5,627-5,684.
#ifndef TC_BCAST_COPIES
#define TC_BCAST_COPIES 4
#endif
#ifndef TC_BCAST_WINDOW
#define TC_BCAST_WINDOW 8192
#endif
#ifndef TC_BCAST_NT_SRC
#define TC_BCAST_NT_SRC 0
#endif
struct BcastArgs {
    const char* src;
    char* dst[TC_MAX_K];
    int K, es;
    int64_t nbytes;
    int64_t nchunk, window;  // chunks of TC_EW_THREADS slots; chunks per window (>= 1)
    int C, groups;           // copies per workgroup; ceil(K / C)
};

// K = 1 with 16-byte aligned buffers, a plain copy: every workgroup copies
// one chunk of TC_EW_THREADS slots, read once (non-temporal).  Its
// arguments are only what that needs, so the load issues after one round
// of scalar loads, where the general kernel's prologue waits on a chain of
// them.  Measured on MI355X, 1 GiB: 6.17-6.24 TB/s through the general
// kernel, 6.44-6.52 through this one; at K = 2 and 4 the same shape (all
// copies per workgroup, non-temporal source) was 1.6-2.2% slower than the
// general kernel.  Lanes past the last whole slot copy that slot again
// (the same bytes to the same place), so no branch holds the loads back;
// the host takes this kernel only with at least one whole slot.  Workgroup
// 0 also copies the bytes after the last whole slot.
struct CopyArgs {
    const u4* src;
    u4* dst;
    int64_t nvec;    // whole 16-byte slots (>= 1)
    int64_t nbytes;  // all bytes (tail: nvec * 16 .. nbytes)
    int es;
};

__global__ __launch_bounds__(TC_EW_THREADS) void copy_kernel(CopyArgs a) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * TC_EW_THREADS + threadIdx.x;
    const int64_t v = i < a.nvec ? i : a.nvec - 1;
    __builtin_nontemporal_store(__builtin_nontemporal_load(a.src + v), a.dst + v);
    if (blockIdx.x == 0)
        for (int64_t b = a.nvec * 16 + threadIdx.x * a.es; b < a.nbytes; b += TC_EW_THREADS * a.es) {
            const char* sp = reinterpret_cast<const char*>(a.src) + b;
            char* dp = reinterpret_cast<char*>(a.dst) + b;
            if (a.es == 4) *reinterpret_cast<uint32_t*>(dp) = *reinterpret_cast<const uint32_t*>(sp);
            else *reinterpret_cast<uint16_t*>(dp) = *reinterpret_cast<const uint16_t*>(sp);
        }
}

template <bool VEC>
__global__ __launch_bounds__(TC_EW_THREADS) void bcast_kernel(BcastArgs a) {
    if (VEC) {
        const int64_t nvec = a.nbytes / 16;
        if (a.nchunk > 0) {
            const int64_t b = blockIdx.x;
            const int64_t per_window = a.window * a.groups;  // every window but the last is full
            const int64_t w = b / per_window;
            const int64_t rest = a.nchunk - w * a.window;
            const int64_t wlen = rest < a.window ? rest : a.window;
            const int64_t r = b - w * per_window;
            const int64_t cg = r / wlen;
            const int64_t v = (w * a.window + (r - cg * wlen)) * TC_EW_THREADS + threadIdx.x;
            const int k0 = static_cast<int>(cg) * a.C;
            const int k1 = k0 + a.C < a.K ? k0 + a.C : a.K;
            if (v < nvec) {
                const u4* sp = reinterpret_cast<const u4*>(a.src) + v;
                const u4 x = TC_BCAST_NT_SRC ? __builtin_nontemporal_load(sp) : *sp;
                for (int k = k0; k < k1; ++k) __builtin_nontemporal_store(x, reinterpret_cast<u4*>(a.dst[k]) + v);
            }
        }
        if (blockIdx.x == gridDim.x - 1)
            for (int64_t b = nvec * 16 + threadIdx.x * a.es; b < a.nbytes; b += TC_EW_THREADS * a.es)
                for (int k = 0; k < a.K; ++k) {
                    if (a.es == 4) *reinterpret_cast<uint32_t*>(a.dst[k] + b) = *reinterpret_cast<const uint32_t*>(a.src + b);
                    else *reinterpret_cast<uint16_t*>(a.dst[k] + b) = *reinterpret_cast<const uint16_t*>(a.src + b);
                }
    } else {
        const int64_t stride = static_cast<int64_t>(gridDim.x) * TC_EW_THREADS;
        const int64_t t0 = static_cast<int64_t>(blockIdx.x) * TC_EW_THREADS + threadIdx.x;
        for (int64_t e = t0; e * a.es < a.nbytes; e += stride)
            for (int k = 0; k < a.K; ++k) {
                if (a.es == 4) reinterpret_cast<uint32_t*>(a.dst[k])[e] = reinterpret_cast<const uint32_t*>(a.src)[e];
                else reinterpret_cast<uint16_t*>(a.dst[k])[e] = reinterpret_cast<const uint16_t*>(a.src)[e];
            }
    }
}

template <int K, typename T>
hipError_t run_sgd(float* const* x, const void* const* g, float eta, int k_total, int64_t n, bool vec, hipStream_t s) {
    SgdArgs<K, T> a{};
    for (int q = 0; q < k_total; ++q) {
        a.x[q] = x[q];
        a.g[q] = static_cast<const T*>(g[q]);
    }
    a.eta = eta;
    a.k_total = k_total;
    return launch<K, T, easgd_unroll(K)>(a, n, vec, 4, s);
}

template <int K, typename T>
hipError_t run_sync(float* const* x, void* const* g, float step, int broadcast, int k_total, int64_t n, bool vec,
                    hipStream_t s) {
    SyncArgs<K, T> a{};
    for (int q = 0; q < k_total; ++q) {
        a.x[q] = x[q];
        a.g[q] = static_cast<T*>(g[q]);
    }
    a.step = step;
    a.broadcast = broadcast;
    a.k_total = k_total;
    return launch<K, T, easgd_unroll(K)>(a, n, vec, 4, s);
}

template <int K, typename T>
hipError_t run_async(float* const* x, float* xc, const int32_t* order, int R, float alpha, int k_total, int64_t n,
                     bool vec, hipStream_t s) {
    AsyncArgsT<K, T> a{};
    for (int q = 0; q < k_total; ++q) a.x[q] = x[q];
    for (int r = 0; r < R; ++r) a.order[r] = static_cast<uint8_t>(order[r]);
    a.xc = xc;
    a.R = R;
    a.alpha = alpha;
    a.k_total = k_total;
    return launch<K, T, easgd_unroll(K)>(a, n, vec, 4, s);
}

template <typename T>
hipError_t dispatch_sgd(int K, float* const* x, const void* const* g, float eta, int64_t n, bool vec, hipStream_t s) {
    switch (K) {
#define TC_CASE(k) \
    case k: return run_sgd<k, T>(x, g, eta, K, n, vec, s);
        TC_FOR_K(TC_CASE)
#undef TC_CASE
        default: return run_sgd<TC_MAX_K, T>(x, g, eta, K, n, vec, s);
    }
}

template <typename T>
hipError_t dispatch_sync(int K, float* const* x, void* const* g, float step, int broadcast, int64_t n, bool vec,
                         hipStream_t s) {
    switch (K) {
#define TC_CASE(k) \
    case k: return run_sync<k, T>(x, g, step, broadcast, K, n, vec, s);
        TC_FOR_K(TC_CASE)
#undef TC_CASE
        default: return run_sync<TC_MAX_K, T>(x, g, step, broadcast, K, n, vec, s);
    }
}

hipError_t dispatch_async(int K, float* const* x, float* xc, const int32_t* order, int R, float alpha, int64_t n,
                          bool vec, hipStream_t s) {
    switch (K) {
#define TC_CASE(k) \
    case k: return run_async<k, float>(x, xc, order, R, alpha, K, n, vec, s);
        TC_FOR_K(TC_CASE)
#undef TC_CASE
        default: return run_async<TC_MAX_K, float>(x, xc, order, R, alpha, K, n, vec, s);
    }
}

}  // namespace

hipError_t launch_sgd(int K, float* const* x, const void* const* g, int g_dtype, float eta, int64_t n, bool vector_ok,
                      hipStream_t stream) {
    if (g_dtype == TC_BF16) return dispatch_sgd<uint16_t>(K, x, g, eta, n, vector_ok, stream);
    return dispatch_sgd<float>(K, x, g, eta, n, vector_ok, stream);
}

hipError_t launch_sync_sgd(int K, float* const* x, void* const* g, int g_dtype, float eta, float rescale, int broadcast,
                           int64_t n, bool vector_ok, hipStream_t stream) {
    const float step = eta * rescale;  // one binary32 rounding, on the host
    if (g_dtype == TC_BF16) return dispatch_sync<uint16_t>(K, x, g, step, 0, n, vector_ok, stream);
    return dispatch_sync<float>(K, x, g, step, broadcast, n, vector_ok, stream);
}

hipError_t launch_elastic_async(int K, float* const* x, float* xc, const int32_t* order, int R, float alpha,
                                int64_t n, bool vector_ok, hipStream_t stream) {
    return dispatch_async(K, x, xc, order, R, alpha, n, vector_ok, stream);
}

hipError_t launch_broadcast(int K, const void* src, void* const* dst, int es, int64_t n, bool vector_ok,
                            hipStream_t stream) {
    BcastArgs a{};
    a.src = static_cast<const char*>(src);
    for (int k = 0; k < K; ++k) a.dst[k] = static_cast<char*>(dst[k]);
    a.K = K;
    a.es = es;
    a.nbytes = n * es;
    if (vector_ok && K == 1 && a.nbytes >= 16) {
        CopyArgs c{static_cast<const u4*>(src), static_cast<u4*>(dst[0]), a.nbytes / 16, a.nbytes, es};
        dim3 grid(static_cast<unsigned>((c.nvec + TC_EW_THREADS - 1) / TC_EW_THREADS));
        hipLaunchKernelGGL(copy_kernel, grid, dim3(TC_EW_THREADS), 0, stream, c);
    } else if (vector_ok) {
        a.nchunk = (a.nbytes / 16 + TC_EW_THREADS - 1) / TC_EW_THREADS;
        a.window = a.nchunk < TC_BCAST_WINDOW ? (a.nchunk > 0 ? a.nchunk : 1) : TC_BCAST_WINDOW;
        a.C = TC_BCAST_COPIES < K ? TC_BCAST_COPIES : K;
        a.groups = (K + a.C - 1) / a.C;
        const int64_t blocks = a.nchunk * a.groups;
        dim3 grid(static_cast<unsigned>(blocks > 0 ? blocks : 1));
        hipLaunchKernelGGL((bcast_kernel<true>), grid, dim3(TC_EW_THREADS), 0, stream, a);
    } else {
        dim3 grid(static_cast<unsigned>(grid_for(n, 1)));
        hipLaunchKernelGGL((bcast_kernel<false>), grid, dim3(TC_EW_THREADS), 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_reduce(int K, const void* const* in, int in_dtype, float* out, int op, int64_t n, bool vector_ok,
                         hipStream_t stream) {
    if (in_dtype == TC_BF16) return dispatch_reduce<uint16_t>(K, in, out, op, n, vector_ok, stream);
    return dispatch_reduce<float>(K, in, out, op, n, vector_ok, stream);
}

hipError_t launch_easgd(int K, float* const* x, const void* const* g, int g_dtype, float* xc, float* out, int op,
                        float eta, float rho, int64_t n, bool vector_ok, hipStream_t stream) {
    if (g_dtype == TC_BF16) return dispatch_easgd<uint16_t>(K, x, g, xc, out, op, eta, rho, n, vector_ok, stream);
    return dispatch_easgd<float>(K, x, g, xc, out, op, eta, rho, n, vector_ok, stream);
}

}  // namespace tc
