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
#include <type_traits>

#include "tc_internal.h"

#ifndef TC_TEASGD_CSHARE
#define TC_TEASGD_CSHARE 1
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

// Two-input DPP: lanes in the enabled banks (groups of 4 lanes of a row)
// take CTRL's source lane from src, the others keep old.
template <int CTRL, int BANKS>
__device__ __forceinline__ float dpp_banks(float old, float src) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                                  __builtin_bit_cast(int, src), CTRL, 0xF, BANKS,
                                                                  false));
}

// Split group sum of the four components of v over each aligned group of P
// (>= 4) lanes.  Partner l^1 exchanges halves (lane bit 0 keeps components
// {0,1} or {2,3}), partner l^2 exchanges quarters (bit 1 picks one of the
// two), so after two steps each lane carries one component, and the
// remaining steps add whole groups: l^4 (row rotates by 12 and by 4, each
// written to the banks it serves), l^8 (row rotate by 8), l^16, l^32.  The
// terms meet in the order of the pairwise tree, as in group_sum; each lane
// ends with component comp_of_lane(l) of the group's sum, a quarter of the
// work of summing all four components in every lane.
__device__ __forceinline__ int comp_of_lane(int lane) { return ((lane & 1) << 1) | ((lane >> 1) & 1); }

template <int P>
__device__ __forceinline__ float split_group_sum(f4 v, int lane) {
    static_assert(P >= 4, "two split steps need four lanes");
    const bool b = lane & 1, c = (lane >> 1) & 1;
    const float k0 = b ? v.z : v.x, k1 = b ? v.w : v.y;      // kept half
    const float s0 = b ? v.x : v.z, s1 = b ? v.y : v.w;      // half for the partner
    const float w0 = k0 + dpp<0xB1>(s0), w1 = k1 + dpp<0xB1>(s1);
    float u = (c ? w1 : w0) + dpp<0x4E>(c ? w0 : w1);
    if constexpr (P >= 8) {
        // lane ^ 4: banks 0 and 2 read lane + 4 (rotate by 12), banks 1 and 3
        // read lane - 4 (rotate by 4)
        const float t = dpp_banks<0x12C, 0x5>(u, u);
        u = u + dpp_banks<0x124, 0xA>(t, u);
    }
    if constexpr (P >= 16) u = u + dpp<0x128>(u);  // row_ror:8 = lane ^ 8
    if constexpr (P >= 32) u = u + __shfl_xor(u, 16, 64);
    if constexpr (P >= 64) u = u + __shfl_xor(u, 32, 64);
    return u;
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

// Stores with explicit cache-policy bits (bit 0 sc0, bit 1 nt, bit 4 sc1) as
// raw buffer stores when offsets are 32-bit; AUX < 0 keeps the plain
// non-temporal global store.  Measured on MI355X with a 1 GiB copy between
// calls (so that no call finds its output in the 256 MB last-level cache):
// sc1 on the reduction's output -3% to +3% by group, on the step's center
// +0 to +2%, on the workers and center together level; plain stores (0)
// lost 13-16% on the step.  Called back to back without that copy, sc1 on
// the reduction's output looked 4% faster on the groups whose output fits
// in that cache: the output stayed there from one call to the next.  All
// three keep non-temporal stores.
#ifndef TC_TRD_STORE_AUX
#define TC_TRD_STORE_AUX -1
#endif
#ifndef TC_TEA_X_STORE_AUX
#define TC_TEA_X_STORE_AUX -1
#endif
#ifndef TC_TEA_C_STORE_AUX
#define TC_TEA_C_STORE_AUX -1
#endif
template <int AUX, typename I>
__device__ __forceinline__ void store_slot_pol(float* p, I s, f4 v) {
    if constexpr (AUX >= 0 && sizeof(I) == 4) {
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(p, static_cast<short>(0), -1, 0x00020000);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), r, s * 16u, 0, AUX);
    } else {
        store_slot(p, s, v);
    }
}
template <int AUX, typename I>
__device__ __forceinline__ void store_elem_pol(float* p, I s, int comp, float v) {  // component comp of slot s
    if constexpr (AUX >= 0 && sizeof(I) == 4) {
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(p, static_cast<short>(0), -1, 0x00020000);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, s * 16u + static_cast<uint32_t>(comp) * 4u, 0, AUX);
    } else {
        __builtin_nontemporal_store(v, reinterpret_cast<float*>(reinterpret_cast<char*>(p) + s * I(16)) + comp);
    }
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

// s / K, correctly rounded.  When K = P (a power of two) 1/K is exact, so
// the product with it rounds the same exact quotient: one multiply instead
// of the division sequence.  K is uniform, so the branch is too.
template <int P>
__device__ __forceinline__ float div_k(float s, int K) {
    return K == P ? s * (1.0f / P) : s / static_cast<float>(K);
}
template <int P>
__device__ __forceinline__ f4 div_k(f4 s, int K) {
    return K == P ? s * f4(1.0f / P) : s / f4(static_cast<float>(K));
}

// First slot of this lane: a workgroup covers 4*U*(64/P) consecutive
// slots, each wave U*(64/P) of them, so the single-stream outputs (the
// reduction, the center) leave every wave as >= 128 contiguous bytes.
template <int P, int U, typename I>
__device__ __forceinline__ I first_slot() {
    constexpr int SPW = 64 / P;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t b = tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x);
    return static_cast<I>(b) * (4 * U * SPW) + static_cast<I>(wave * U * SPW + lane / P);
}

// ------------------------------------------------------------- reduce

template <typename T>
struct TReduceArgs {
    const T* in;  // tensor layout, K copies
    float* out;   // N values
    int64_t nslot, n;
    int K, op;
};

// Two consecutive bfloat16 slots (copies s and s + 1 of one slot, s even,
// 16-byte aligned) summed component-wise: the first level of the pairwise
// tree, taken inside the lane.
template <typename I>
__device__ __forceinline__ f4 load_pair_sum(const uint16_t* p, I s) {
    const u4 w = __builtin_nontemporal_load(reinterpret_cast<const u4*>(reinterpret_cast<const char*>(p) + s * I(8)));
    const f4 lo{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u), __uint_as_float(w.y << 16),
                __uint_as_float(w.y & 0xffff0000u)};
    const f4 hi{__uint_as_float(w.z << 16), __uint_as_float(w.z & 0xffff0000u), __uint_as_float(w.w << 16),
                __uint_as_float(w.w & 0xffff0000u)};
    return lo + hi;
}

// The trailing partial slot (the last N % 4 elements), element by element.
template <int P, typename T>
__device__ __forceinline__ void tensor_reduce_tail(const TReduceArgs<T>& a) {
    const int K = a.K;
    const int64_t e = 4 * a.nslot + threadIdx.x;
    if (e < a.n) {
        float t[P];
#pragma unroll
        for (int q = 0; q < P; ++q) t[q] = q < K ? load_elem(a.in, (a.nslot * K + q) * 4 + (e & 3)) : 0.0f;
        float s = Tree<P>::sum(t);
        if (a.op == TC_AVG) s = div_k<P>(s, K);
        a.out[e] = s;
    }
}

// P: K rounded up to a power of two.  One lane per copy (L = P lanes per
// slot), or, for bfloat16 with K even (PAIR), one lane per two copies
// (L = P / 2): each lane loads 16 bytes and adds its pair first, which is
// the tree's first level, so the butterfly over the L lanes finishes the
// same sum in one fewer step with half the lanes.
template <int P, typename T, int U, typename I, bool PAIR>
__global__ __launch_bounds__(256) void tensor_reduce_kernel(TReduceArgs<T> a) {
    constexpr int L = PAIR ? P / 2 : P;
    constexpr int SPW = 64 / L;  // slots per wave and unroll step
    const int K = a.K;
    const int i = threadIdx.x % L;
    const I j0 = first_slot<L, U, I>();
    const I nslot = static_cast<I>(a.nslot);
    f4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        if constexpr (PAIR)
            v[u] = (j < nslot && 2 * i < K) ? load_pair_sum(a.in, j * I(K) + I(2 * i)) : f4(0.0f);
        else
            v[u] = (j < nslot && i < K) ? load_slot(a.in, j * I(K) + I(i)) : f4(0.0f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        if constexpr (L >= 4) {
            // lanes 0-3 of the group hold one component each
            float s = split_group_sum<L>(v[u], threadIdx.x);
            if (a.op == TC_AVG) s = div_k<P>(s, K);
            if (j < nslot && i < 4) store_elem_pol<TC_TRD_STORE_AUX, I>(a.out, j, comp_of_lane(i), s);
        } else {
            f4 s = group_sum4<L>(v[u]);
            if (a.op == TC_AVG) s = div_k<P>(s, K);
            if (j < nslot && i == 0) store_slot_pol<TC_TRD_STORE_AUX, I>(a.out, j, s);
        }
    }
    if (blockIdx.x == gridDim.x - 1) tensor_reduce_tail<P, T>(a);
}

// The reduction staged through LDS, as the fused step is: a workgroup's S
// slots (S K <= 256 R pieces) are read piece after piece, every lane active,
// and each slot group's split butterfly runs on its copies in LDS, with the
// slot kernel's operations and order.  It serves bfloat16 copies at K not a
// power of two (P >= 8), where the slot kernel reads one 8-byte copy per
// lane (odd K) or idles lanes: the pieces come in two to a lane with 16-byte
// loads (S even keeps the workgroup's first piece 16-byte aligned), and each
// lane adds copies 2i and 2i + 1, the pairwise tree's first level, before a
// butterfly over P / 2 lanes.  Measured on MI355X, ResNet-50 group, against
// the slot kernels: odd K = 5 to 13 3.3-4.5 -> 6.0-6.4 TB/s, K = 17 to 63
// 1.9-2.7 -> 5.1-6.4; even K = 6 to 48 +3-32%; 8 rounds of 256 pieces per
// workgroup against 2, 4, 6, 12 and 16.  For binary32 copies (P >= 32) the
// staged form measured 5-18% slower with one copy per lane, -4 to +2.5%
// with pairs, and is not used.
#ifndef TC_TRD_STAGED_R
#define TC_TRD_STAGED_R 8
#endif
#ifndef TC_TRD_STAGED
#define TC_TRD_STAGED 1
#endif
#ifndef TC_TRD_STAGED_MINP
#define TC_TRD_STAGED_MINP 8
#endif
template <int P, typename T, int R, typename I, bool PAIR>
__global__ __launch_bounds__(256) void tensor_reduce_staged_kernel(TReduceArgs<T> a, int S) {
    constexpr int L = PAIR ? P / 2 : P;  // lanes per slot group
    constexpr int SPB = 256 / L;         // slot groups per pass
    constexpr int UC = 2 * R * L / P;    // passes: S K <= 256 R and K > P / 2 give S < UC SPB
    using V = typename std::conditional<sizeof(T) == 4, u4, u2>::type;  // a stored piece
    __shared__ V s_v[256 * R];
    const int K = a.K;
    const I s0 = static_cast<I>(tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x)) * I(S);
    const I nslot = static_cast<I>(a.nslot);
    const int ns = s0 < nslot ? static_cast<int>(nslot - s0 < I(S) ? nslot - s0 : I(S)) : 0;
    const int np = ns * K;
    const I p0 = s0 * I(K);
    if constexpr (sizeof(T) == 2) {
        // 8-byte pieces two to a lane, one 16-byte load (S is even, so the
        // workgroup's first piece is 16-byte aligned)
        constexpr int R2 = (R + 1) / 2;
        u4 w[R2];
        const char* base = reinterpret_cast<const char*>(a.in) + p0 * I(8);
#pragma unroll
        for (int u = 0; u < R2; ++u) {
            const int q = 2 * (threadIdx.x + u * 256);
            if (q + 1 < np) w[u] = __builtin_nontemporal_load(reinterpret_cast<const u4*>(base + q * 8));
            else if (q < np) {
                const u2 h = __builtin_nontemporal_load(reinterpret_cast<const u2*>(base + q * 8));
                w[u] = u4{h.x, h.y, 0u, 0u};
            }
        }
#pragma unroll
        for (int u = 0; u < R2; ++u) {
            const int q = 2 * (threadIdx.x + u * 256);
            if (q < np) s_v[q] = V{w[u].x, w[u].y};
            if (q + 1 < np) s_v[q + 1] = V{w[u].z, w[u].w};
        }
    } else {
        V v[R];
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int q = threadIdx.x + u * 256;
            if (q < np)
                v[u] = __builtin_nontemporal_load(
                    reinterpret_cast<const V*>(reinterpret_cast<const char*>(a.in) + (p0 + I(q)) * I(sizeof(V))));
        }
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int q = threadIdx.x + u * 256;
            if (q < np) s_v[q] = v[u];
        }
    }
    __syncthreads();
    auto piece = [&](int q) -> f4 {
        const V w = s_v[q];
        if constexpr (sizeof(T) == 4)
            return f4{__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z), __uint_as_float(w.w)};
        else
            return f4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u), __uint_as_float(w.y << 16),
                      __uint_as_float(w.y & 0xffff0000u)};
    };
    const int i = threadIdx.x % L;
#pragma unroll
    for (int u = 0; u < UC; ++u) {
        if (u * SPB >= ns) break;  // the same for the whole workgroup
        const int jl = u * SPB + static_cast<int>(threadIdx.x) / L;
        const bool slot = jl < ns;
        f4 x = f4(0.0f);
        if constexpr (PAIR) {
            // copies 2i and 2i + 1 added in the lane: the pairwise tree's
            // first level (a missing last copy is the tree's +0 padding)
            const f4 lo = slot && 2 * i < K ? piece(jl * K + 2 * i) : f4(0.0f);
            const f4 hi = slot && 2 * i + 1 < K ? piece(jl * K + 2 * i + 1) : f4(0.0f);
            x = lo + hi;
        } else if (slot && i < K) {
            x = piece(jl * K + i);
        }
        float r = split_group_sum<L>(x, threadIdx.x);
        if (a.op == TC_AVG) r = div_k<P>(r, K);
        if (slot && i < 4) store_elem_pol<TC_TRD_STORE_AUX, I>(a.out, s0 + I(jl), comp_of_lane(i), r);
    }
    if (blockIdx.x == gridDim.x - 1) tensor_reduce_tail<P, T>(a);
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
    float* out;      // RED: N values, the SUM (op TC_SUM) or AVG of the K gradients
    int op;
};

// The trailing partial slot (the last N % 4 elements), element by element.
template <int P, typename T, bool RED>
__device__ __forceinline__ void tensor_easgd_tail(const TEasgdArgs<T>& a) {
    const int K = a.K;
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
        if constexpr (RED) {
            // the gradients again, once the center's terms are summed:
            // holding both sets of P terms would size every lane of the
            // kernel for them
            float t[P];
#pragma unroll
            for (int q = 0; q < P; ++q) t[q] = q < K ? load_elem(a.g, (a.nslot * K + q) * 4 + (e & 3)) : 0.0f;
            float r = Tree<P>::sum(t);
            if (a.op == TC_AVG) r = div_k<P>(r, K);
            a.out[e] = r;
        }
    }
}

// A wave of the step covers WS = U * 64 / P consecutive slots.  At P >= 16
// that is at most 8 slots, 128 bytes of the center, which U instructions of
// 64 / P slots each would read and write in pieces of 16 to 64 bytes; the
// center is then read by one instruction (lane m < WS takes slot m of the
// wave) and handed to the slot groups with cross-lane reads, and the new
// center gathered back into lanes 0 .. WS - 1 for one store.
__device__ __forceinline__ f4 shfl4(f4 v, int src) {
    return f4{__shfl(v.x, src, 64), __shfl(v.y, src, 64), __shfl(v.z, src, 64), __shfl(v.w, src, 64)};
}

#ifndef TC_TEA_RED_GATHER
#define TC_TEA_RED_GATHER 1
#endif
#ifndef TC_TEA_RED_SPLIT
#define TC_TEA_RED_SPLIT 1
#endif
// RED: the step fused with the reduction of the gradients it reads, by the
// reduction kernel's own butterflies and quotient (bit for bit its result).
template <int P, typename T, int U, typename I, bool RED>
__global__ __launch_bounds__(256) void tensor_easgd_kernel(TEasgdArgs<T> a) {
    constexpr int SPW = 64 / P;
    constexpr int WS = U * SPW;
    constexpr bool kShare = P >= 16 && TC_TEASGD_CSHARE;
    const int K = a.K;
    const int i = threadIdx.x % P;
    const int lane = threadIdx.x & 63;
    const I j0 = first_slot<P, U, I>();
    const I jw = j0 - static_cast<I>(lane / P);  // the wave's first slot
    const I nslot = static_cast<I>(a.nslot);
    f4 x[U], g[U], c[U];
    if constexpr (kShare) {
        const I jm = jw + static_cast<I>(lane % WS);
        const f4 cw = jm < nslot ? load_slot(a.xc, jm) : f4(0.0f);
#pragma unroll
        for (int u = 0; u < U; ++u) c[u] = shfl4(cw, lane / P + u * SPW);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        const bool slot = j < nslot;
        if constexpr (!kShare) c[u] = slot ? load_slot(a.xc, j) : f4(0.0f);
        const bool live = slot && i < K;
        x[u] = live ? load_slot(a.x, j * I(K) + I(i)) : f4(0.0f);
        g[u] = live ? load_slot(a.g, j * I(K) + I(i)) : f4(0.0f);
    }
    const f4 rho = f4(a.rho), neg_eta = f4(-a.eta), alpha = f4(a.a);
    f4 cn[U];
    f4 rout = f4(0.0f);  // RED at P >= 16: lane m < WS gathers the output of the wave's slot m
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        const bool live = j < nslot && i < K;
        const f4 d = live ? x[u] - c[u] : f4(0.0f);
        const f4 xn = fma4(neg_eta, fma4(rho, d, g[u]), x[u]);
        cn[u] = fma4(alpha, group_sum4<P>(d), c[u]);
        if (live) store_slot_pol<TC_TEA_X_STORE_AUX, I>(a.x, j * I(K) + I(i), xn);
        if (!kShare && j < nslot && i == 0) store_slot_pol<TC_TEA_C_STORE_AUX, I>(a.xc, j, cn[u]);
        if constexpr (RED) {
            // the gradients of lanes past K, and of slots past the end, are +0
            if constexpr (kShare && TC_TEA_RED_GATHER) {
                // the slot groups' sums gathered like the center, so that the
                // wave writes its WS slots of the output with one store, and
                // the AVG quotient taken once, after the gather.  The split
                // butterfly leaves lane c' of a slot group with component
                // comp_of_lane(c') (a self-inverse map of its two low bits);
                // the gather reads the four components from those lanes.
#if TC_TEA_RED_SPLIT
                const float r1 = split_group_sum<P>(g[u], threadIdx.x);
                const int base = (lane % SPW) * P;
                const f4 t{__shfl(r1, base, 64), __shfl(r1, base + 2, 64), __shfl(r1, base + 1, 64),
                           __shfl(r1, base + 3, 64)};
#else
                const f4 t = shfl4(group_sum4<P>(g[u]), (lane % SPW) * P);
#endif
                if (lane / SPW == u) rout = t;
            } else if constexpr (P >= 4) {
                float r = split_group_sum<P>(g[u], threadIdx.x);
                if (a.op == TC_AVG) r = div_k<P>(r, K);
                if (j < nslot && i < 4) store_elem_pol<TC_TRD_STORE_AUX, I>(a.out, j, comp_of_lane(i), r);
            } else {
                f4 r = group_sum4<P>(g[u]);
                if (a.op == TC_AVG) r = div_k<P>(r, K);
                if (j < nslot && i == 0) store_slot_pol<TC_TRD_STORE_AUX, I>(a.out, j, r);
            }
        }
    }
    if constexpr (kShare) {
        // lane m < WS stores slot jw + m, whose new center slot group m % SPW
        // computed in pass m / SPW
        f4 out = f4(0.0f);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const f4 t = shfl4(cn[u], (lane % SPW) * P);
            if (lane / SPW == u) out = t;
        }
        if (lane < WS && jw + static_cast<I>(lane) < nslot)
            store_slot_pol<TC_TEA_C_STORE_AUX, I>(a.xc, jw + static_cast<I>(lane), out);
        if constexpr (RED && TC_TEA_RED_GATHER) {
            if (a.op == TC_AVG) rout = div_k<P>(rout, K);
            if (lane < WS && jw + static_cast<I>(lane) < nslot)
                store_slot_pol<TC_TRD_STORE_AUX, I>(a.out, jw + static_cast<I>(lane), rout);
        }
    }
    if (blockIdx.x == gridDim.x - 1) tensor_easgd_tail<P, T, RED>(a);
}

// When K is not a power of two, P - K of every P lanes of the slot mapping
// idle in each load and store.  The staged form moves a workgroup's S slots
// (S K <= 256 R pieces) between HBM and LDS piece after piece, every lane
// active but in a last partial round, and runs each
// slot group's arithmetic on its copies in LDS: the same operations on the
// same values in the same order as tensor_easgd_kernel, so the results are
// bit-identical.  The sums over a slot's copies take the split butterfly
// (each of a group's first four lanes ends with one component).  A slot
// group's center slot is read by all of its lanes and then overwritten, one
// component each, by its first four; the group lies in one wave, whose
// instructions run in order, so every lane reads it first.
#ifndef TC_TEA_STAGED_MINP
#define TC_TEA_STAGED_MINP 32
#endif
#ifndef TC_TEA_STAGED_R
#define TC_TEA_STAGED_R 2
#endif
template <int P, typename T, int R, typename I, bool RED>
__global__ __launch_bounds__(256) void tensor_easgd_staged_kernel(TEasgdArgs<T> a, int S) {
    constexpr int SPB = 256 / P;  // slot groups per pass
    constexpr int UC = 2 * R;     // passes: S K <= 256 R and K > P / 2 give S < UC SPB
    __shared__ f4 s_x[256 * R], s_g[256 * R], s_c[UC * SPB], s_r[RED ? UC * SPB : 1];
    const int K = a.K;
    const I s0 = static_cast<I>(tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x)) * I(S);
    const I nslot = static_cast<I>(a.nslot);
    const int ns = s0 < nslot ? static_cast<int>(nslot - s0 < I(S) ? nslot - s0 : I(S)) : 0;
    const int np = ns * K;
    const I p0 = s0 * I(K);
    f4 vx[R], vg[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int q = threadIdx.x + u * 256;
        if (q < np) {
            vx[u] = load_slot(a.x, p0 + I(q));
            vg[u] = load_slot(a.g, p0 + I(q));
        }
    }
    if (static_cast<int>(threadIdx.x) < ns) s_c[threadIdx.x] = load_slot(a.xc, s0 + I(threadIdx.x));
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int q = threadIdx.x + u * 256;
        if (q < np) {
            s_x[q] = vx[u];
            s_g[q] = vg[u];
        }
    }
    __syncthreads();
    const int i = threadIdx.x % P;
    const f4 rho = f4(a.rho), neg_eta = f4(-a.eta);
#pragma unroll
    for (int u = 0; u < UC; ++u) {
        if (u * SPB >= ns) break;  // the same for the whole workgroup
        const int jl = u * SPB + static_cast<int>(threadIdx.x) / P;
        const bool slot = jl < ns, live = slot && i < K;
        const int q = jl * K + i;
        const f4 x = live ? s_x[q] : f4(0.0f), g = live ? s_g[q] : f4(0.0f);
        const f4 c = slot ? s_c[jl] : f4(0.0f);
        const f4 d = live ? x - c : f4(0.0f);
        const f4 xn = fma4(neg_eta, fma4(rho, d, g), x);
        const int m = comp_of_lane(i);
        const float sd = split_group_sum<P>(d, threadIdx.x);
        const float cm = m == 0 ? c.x : m == 1 ? c.y : m == 2 ? c.z : c.w;
        if (live) s_x[q] = xn;
        if (slot && i < 4) reinterpret_cast<float*>(s_c)[jl * 4 + m] = __builtin_fmaf(a.a, sd, cm);
        if constexpr (RED) {
            // the gradients of lanes past K are +0
            float r = split_group_sum<P>(g, threadIdx.x);
            if (a.op == TC_AVG) r = div_k<P>(r, K);
            if (slot && i < 4) reinterpret_cast<float*>(s_r)[jl * 4 + m] = r;
        }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int q = threadIdx.x + u * 256;
        if (q < np) store_slot_pol<TC_TEA_X_STORE_AUX, I>(a.x, p0 + I(q), s_x[q]);
    }
    if (static_cast<int>(threadIdx.x) < ns) {
        store_slot_pol<TC_TEA_C_STORE_AUX, I>(a.xc, s0 + I(threadIdx.x), s_c[threadIdx.x]);
        if constexpr (RED) store_slot_pol<TC_TRD_STORE_AUX, I>(a.out, s0 + I(threadIdx.x), s_r[threadIdx.x]);
    }
    if (blockIdx.x == gridDim.x - 1) tensor_easgd_tail<P, T, RED>(a);
}

// ------------------------------------------ sgd / sync / async / broadcast

template <typename T>
struct TStepArgs {
    float* x;       // tensor layout, K copies
    T* g;           // tensor layout, K copies (gradients)
    float* xc;      // N values (async exchange)
    int64_t nslot, n;
    float s0, s1;   // sgd: eta; sync: eta*rescale; async: alpha
    int K, flag;    // sync: broadcast the sum into g
    uint8_t order[TC_MAX_K];
    int R;
    uint64_t exchanged;  // async: bit w set when worker w is in order[0..R)
};

enum class TOp { Sgd, Sync, Async };

// The trailing partial slot (the last N % 4 elements), element by element.
template <TOp OP, int P, typename T>
__device__ __forceinline__ void tensor_step_tail(const TStepArgs<T>& a) {
    const int K = a.K;
    const int64_t e = 4 * a.nslot + threadIdx.x;
    if (e < a.n) {
        auto idx = [&](int q) { return (a.nslot * K + q) * 4 + (e & 3); };
        if constexpr (OP == TOp::Sgd) {
            for (int q = 0; q < K; ++q)
                a.x[idx(q)] = __builtin_fmaf(-a.s0, load_elem(static_cast<const T*>(a.g), idx(q)), a.x[idx(q)]);
        } else if constexpr (OP == TOp::Sync) {
            float t[P];
#pragma unroll
            for (int q = 0; q < P; ++q) t[q] = q < K ? load_elem(static_cast<const T*>(a.g), idx(q)) : 0.0f;
            const float S = Tree<P>::sum(t);
            for (int q = 0; q < K; ++q) {
                a.x[idx(q)] = __builtin_fmaf(-a.s0, S, a.x[idx(q)]);
                if constexpr (sizeof(T) == 4)
                    if (a.flag) reinterpret_cast<float*>(a.g)[idx(q)] = S;
            }
        } else {
            float c = a.xc[e];
            for (int r = 0; r < a.R; ++r) {
                const int64_t k = idx(a.order[r]);
                const float d = a.x[k] - c;
                c = __builtin_fmaf(a.s0, d, c);
                a.x[k] = __builtin_fmaf(-a.s0, d, a.x[k]);
            }
            a.xc[e] = c;
        }
    }
}




template <TOp OP, int P, typename T, typename I>
__global__ __launch_bounds__(256) void tensor_step_kernel(TStepArgs<T> a) {
    constexpr int SPW = 64 / P;
    const int K = a.K;
    const int i = threadIdx.x % P;
    const I j = first_slot<P, 1, I>();
    const I nslot = static_cast<I>(a.nslot);
    const bool slot = j < nslot;
    const bool live = slot && i < K;
    const I piece = j * I(K) + I(i);
    (void)SPW;
    if constexpr (OP == TOp::Sgd) {
        if (live) {
            const f4 x = load_slot(a.x, piece), g = load_slot(static_cast<const T*>(a.g), piece);
            store_slot(a.x, piece, fma4(f4(-a.s0), g, x));
        }
    } else if constexpr (OP == TOp::Sync) {
        const f4 g = live ? load_slot(static_cast<const T*>(a.g), piece) : f4(0.0f);
        const f4 x = live ? load_slot(a.x, piece) : f4(0.0f);
        const f4 S = group_sum4<P>(g);
        if (live) {
            store_slot(a.x, piece, fma4(f4(-a.s0), S, x));
            if constexpr (sizeof(T) == 4)
                if (a.flag) store_slot(reinterpret_cast<float*>(a.g), piece, S);
        }
    } else {
        // P <= 2: every lane of the slot's group runs the four-wide
        // recurrence over the (at most 2) exchanges, reading the exchanged
        // worker's slot from LDS
        __shared__ f4 s_x[256];
        const f4 x = live ? load_slot(a.x, piece) : f4(0.0f);
        f4 c = slot ? load_slot(a.xc, j) : f4(0.0f);
        s_x[threadIdx.x] = x;
        __syncthreads();
        const int group = threadIdx.x & ~(P - 1);
        f4 d_mine = f4(0.0f);
        bool mine = false;
        for (int r = 0; r < a.R; ++r) {
            const int w = a.order[r];
            const f4 d = s_x[group + w] - c;
            if (w == i) {
                d_mine = d;
                mine = true;
            }
            c = fma4(f4(a.s0), d, c);
        }
        if (live && mine) store_slot(a.x, piece, fma4(f4(-a.s0), d_mine, x));
        if (slot && i == 0) store_slot(a.xc, j, c);
    }
    if (blockIdx.x == gridDim.x - 1) tensor_step_tail<OP, P, T>(a);
}

// The asynchronous exchange at P >= 4.  The center's recurrence over the
// exchanges, c = fma(alpha, x_w - c, c) in order, is four scalar
// recurrences, one per component of a slot: lanes 0-3 of each slot's group
// run them, reading the exchanged worker's component from LDS and writing
// each step's difference to that worker's row of a second LDS array; each
// exchanged worker then takes its difference from its row.  (With all P
// lanes running the four-wide recurrence, the per-slot work grew as K^2:
// ALU-bound from K = 16 on.  Measured on MI355X against that, ResNet-50
// group, R = K: K = 4 +23%, K = 16 +18%, K = 32 +59%, K = 64 +67%, K = 3 and
// 8 level.)  The groups' rows are padded by one slot, so that the active
// lanes of a wave, reading or writing component i of the same worker in
// every group, fall in distinct LDS banks.  A lane takes U = 2 slots, whose
// recurrences interleave: with one, a kernel whose K is below P moved too
// few bytes per wave (measured on MI355X against one slot: K = 3 +17%, K = 5
// +35%, K = 8 +3%, K = 16 +5%, K = 32 +12%, VGG-16 K = 4 -3%; four slots
// measured level or below two).
template <int P, int U, typename I>
__global__ __launch_bounds__(256) void tensor_async_kernel(TStepArgs<float> a) {
    constexpr int SPW = 64 / P;
    constexpr int ROWS = 256 + 256 / P;
    const int K = a.K;
    const int i = threadIdx.x % P;
    const I j0 = first_slot<P, U, I>();
    const I nslot = static_cast<I>(a.nslot);
    __shared__ f4 s_x[U][ROWS];
    __shared__ f4 s_d[U][ROWS];
    const int row0 = (threadIdx.x & ~(P - 1)) + static_cast<int>(threadIdx.x) / P;  // the group's padded row 0
    f4 x[U];
    float c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        const bool slot = j < nslot;
        x[u] = slot && i < K ? load_slot(a.x, j * I(K) + I(i)) : f4(0.0f);
        c[u] = slot && i < 4 ? __builtin_nontemporal_load(a.xc + (j * I(4) + I(i))) : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) s_x[u][row0 + i] = x[u];
    __syncthreads();
    if (i < 4) {
#pragma unroll 4
        for (int r = 0; r < a.R; ++r) {
            const int w = a.order[r];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float d = reinterpret_cast<const float*>(&s_x[u][row0 + w])[i] - c[u];
                reinterpret_cast<float*>(&s_d[u][row0 + w])[i] = d;
                c[u] = __builtin_fmaf(a.s0, d, c[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const I j = j0 + I(u) * SPW;
            if (j < nslot) __builtin_nontemporal_store(c[u], a.xc + (j * I(4) + I(i)));
        }
    }
    __syncthreads();
    if (i < K && ((a.exchanged >> i) & 1)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const I j = j0 + I(u) * SPW;
            if (j < nslot) store_slot(a.x, j * I(K) + I(i), fma4(f4(-a.s0), s_d[u][row0 + i], x[u]));
        }
    }
    if (blockIdx.x == gridDim.x - 1) {  // trailing partial slot, element by element
        const int64_t e = 4 * a.nslot + threadIdx.x;
        if (e < a.n) {
            float ce = a.xc[e];
            for (int r = 0; r < a.R; ++r) {
                const int64_t k = (a.nslot * K + a.order[r]) * 4 + (e & 3);
                const float d = a.x[k] - ce;
                ce = __builtin_fmaf(a.s0, d, ce);
                a.x[k] = __builtin_fmaf(-a.s0, d, a.x[k]);
            }
            a.xc[e] = ce;
        }
    }
}

// The asynchronous exchange staged through LDS (K >= TC_TASYNC_STAGED_K).
// In tensor_async_kernel only lanes 0-3 of each slot group run the
// recurrence, 8 of a wave's 64 lanes at P = 64.  Here a workgroup reads its
// S slots into LDS piece after piece, every lane active, one row of KP = K
// | 1 pieces per slot (an odd row length puts the rows' component i in
// distinct banks), and every lane runs V of the workgroup's 4 S scalar
// recurrences (one per slot and component), updating each exchanged worker
// in place: d = x_w - c, c = fma(alpha, d, c), x_w = fma(-alpha, d, x_w),
// the slot kernel's operations in its order.  The exchanged workers' pieces
// are then written back piece after piece.  The LDS is sized at launch to
// the S rows, S at most 64 and the rows at most 24 KiB, so that more
// workgroups fit per CU.  Measured on MI355X, ResNet-50 group, R = K,
// against the slot kernel: K = 17 +19%, K = 33 2.96 -> 5.09 TB/s, K = 40
// +12% and K = 48 +12% over 64 KiB of rows (+40-45% over the slot kernel),
// K = 56 +24%, K = 64 3.1 -> 3.8; K = 24 -3% and K = 32 -13%.  So it takes
// every K from 33, and K = 17 to 23, where more than a quarter of the slot
// mapping's lanes would idle.  Rows of up to 16, 32 and 64 KiB, and two or
// four recurrences per lane, measured slower.
#ifndef TC_TASYNC_STAGED
#define TC_TASYNC_STAGED 1
#endif
#ifndef TC_TASYNC_STAGED_V
#define TC_TASYNC_STAGED_V 1
#endif
#ifndef TC_TASYNC_STAGED_LDS
#define TC_TASYNC_STAGED_LDS 24576
#endif
template <int V, typename I>
__global__ __launch_bounds__(256) void tensor_async_staged_kernel(TStepArgs<float> a, int S) {
    extern __shared__ f4 s_x[];  // S rows of KP pieces (sized at launch)
    const int K = a.K, KP = K | 1;
    const I s0 = static_cast<I>(tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x)) * I(S);
    const I nslot = static_cast<I>(a.nslot);
    const int ns = s0 < nslot ? static_cast<int>(nslot - s0 < I(S) ? nslot - s0 : I(S)) : 0;
    const int np = ns * K;
    const I p0 = s0 * I(K);
    // pieces in, four loads in flight per lane
    for (int q0 = 0; q0 < np; q0 += 4 * 256) {
        f4 v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int q = q0 + t * 256 + static_cast<int>(threadIdx.x);
            if (q < np) v[t] = load_slot(a.x, p0 + I(q));
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int q = q0 + t * 256 + static_cast<int>(threadIdx.x);
            if (q < np) s_x[(q / K) * KP + q % K] = v[t];
        }
    }
    float c[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
        const int ch = static_cast<int>(threadIdx.x) + v * 256;  // slot ch / 4, component ch % 4
        c[v] = ch < 4 * ns ? __builtin_nontemporal_load(a.xc + ((s0 + I(ch / 4)) * I(4) + I(ch % 4))) : 0.0f;
    }
    __syncthreads();
    float* sx = reinterpret_cast<float*>(s_x);
#pragma unroll 2
    for (int r = 0; r < a.R; ++r) {
        const int w = a.order[r];
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int ch = static_cast<int>(threadIdx.x) + v * 256;
            if (ch < 4 * ns) {
                float* px = sx + ((ch / 4) * KP + w) * 4 + ch % 4;
                const float xw = *px;
                const float d = xw - c[v];
                c[v] = __builtin_fmaf(a.s0, d, c[v]);
                *px = __builtin_fmaf(-a.s0, d, xw);
            }
        }
    }
#pragma unroll
    for (int v = 0; v < V; ++v) {
        const int ch = static_cast<int>(threadIdx.x) + v * 256;
        if (ch < 4 * ns) __builtin_nontemporal_store(c[v], a.xc + ((s0 + I(ch / 4)) * I(4) + I(ch % 4)));
    }
    __syncthreads();
    for (int q = static_cast<int>(threadIdx.x); q < np; q += 256) {
        const int w = q % K;
        if ((a.exchanged >> w) & 1) store_slot(a.x, p0 + I(q), s_x[(q / K) * KP + w]);
    }
    if (blockIdx.x == gridDim.x - 1) tensor_step_tail<TOp::Async, 64, float>(a);  // P is not used by the exchange
}

// Broadcast of one flat buffer into every copy of a tensor-layout buffer.
// A lane takes U slots of its copy (a wave U*64/P adjacent slots) and issues
// all U source loads before its stores.  Measured on MI355X with sources
// rotated so that none is cached between calls (GB/s; ResNet-50 group K = 8 /
// 4 / 16, VGG-16 group K = 4): U = 1 5,087-5,097 / 5,574-5,591 / 4,783-4,818
// / 5,683-5,701; U = 2 5,376-5,404 / 5,969-5,972 / 5,281-5,288 / 6,192;
// U = 4 about 5% below U = 2; U = 8 half of it.
#ifndef TC_TBCAST_UNROLL
#define TC_TBCAST_UNROLL 2
#endif
// K not a power of two takes tensor_bcast_dense_kernel.  Measured on MI355X
// against the slot-group mapping, sources rotated (ResNet-50 group): K = 3
// to 12 +5.5-18%, K = 17 and 33 +31-34% (4.0-4.1 -> 5.3 TB/s), K = 20 to 48
// +8-18%, bfloat16 K = 17 and 33 +50%.
#ifndef TC_TBCAST_DENSE
#define TC_TBCAST_DENSE 1
#endif
template <int P, typename T, int U, typename I>
__global__ __launch_bounds__(256) void tensor_bcast_kernel(const T* src, T* dst, int64_t nslot, int64_t n, int K) {
    constexpr int SB = 4 * sizeof(T);
    constexpr int SPW = 64 / P;
    using V = typename std::conditional<SB == 16, u4, u2>::type;
    const int i = threadIdx.x % P;
    const I j0 = first_slot<P, U, I>();
    const I ns = static_cast<I>(nslot);
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        if (j < ns && i < K) v[u] = *reinterpret_cast<const V*>(reinterpret_cast<const char*>(src) + j * I(SB));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const I j = j0 + I(u) * SPW;
        if (j < ns && i < K)
            __builtin_nontemporal_store(v[u], reinterpret_cast<V*>(reinterpret_cast<char*>(dst) + (j * I(K) + I(i)) * I(SB)));
    }
    if (blockIdx.x == gridDim.x - 1) {
        const int64_t e = 4 * nslot + threadIdx.x;
        if (e < n)
            for (int q = 0; q < K; ++q) dst[(nslot * K + q) * 4 + (e & 3)] = src[e];
    }
}

// The same broadcast with every lane busy when K is not a power of two: the
// destination's whole slots are nslot * K consecutive pieces, lane by lane
// (piece p holds slot p / K of the source), so a wave writes 64 pieces
// whatever K is, where the slot-group mapping leaves P - K of every P lanes
// idle.  A workgroup takes U passes of 256 consecutive pieces.
template <typename T, int U, int PPL, typename I>
__global__ __launch_bounds__(256) void tensor_bcast_dense_kernel(const T* src, T* dst, int64_t nslot, int64_t n,
                                                                 int K) {
    constexpr int SB = 4 * sizeof(T);
    using V = typename std::conditional<SB == 16, u4, u2>::type;
    const I np = static_cast<I>(nslot) * static_cast<I>(K);
    const I p0 = static_cast<I>(tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x)) * I(256 * U) + threadIdx.x;
    const char* sp = reinterpret_cast<const char*>(src);
    char* dp = reinterpret_cast<char*>(dst);
    if constexpr (PPL == 1) {
        V v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const I p = p0 + I(u * 256);
            if (p < np) v[u] = *reinterpret_cast<const V*>(sp + (p / I(K)) * I(SB));
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const I p = p0 + I(u * 256);
            if (p < np) __builtin_nontemporal_store(v[u], reinterpret_cast<V*>(dp + p * I(SB)));
        }
    } else {
        // 8-byte pieces two to a lane (pieces 2q and 2q + 1), stored as one
        // 16-byte granule (the buffer is 16-byte aligned)
        static_assert(SB == 8 && PPL == 2, "two pieces a lane are for 8-byte pieces");
        u2 v[U][2];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const I q = 2 * (p0 + I(u * 256));
            if (q < np) v[u][0] = *reinterpret_cast<const u2*>(sp + (q / I(K)) * I(SB));
            if (q + 1 < np) v[u][1] = *reinterpret_cast<const u2*>(sp + ((q + 1) / I(K)) * I(SB));
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const I q = 2 * (p0 + I(u * 256));
            if (q + 1 < np)
                __builtin_nontemporal_store(u4{v[u][0].x, v[u][0].y, v[u][1].x, v[u][1].y},
                                            reinterpret_cast<u4*>(dp + q * I(SB)));
            else if (q < np)
                __builtin_nontemporal_store(v[u][0], reinterpret_cast<u2*>(dp + q * I(SB)));
        }
    }
    if (blockIdx.x == gridDim.x - 1) {
        const int64_t e = 4 * nslot + threadIdx.x;
        if (e < n)
            for (int q = 0; q < K; ++q) dst[(nslot * K + q) * 4 + (e & 3)] = src[e];
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
    int32_t groups;     // workgroups per chunk, each taking P of the K copies
};

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

// SB source bytes at address S (SB = 16 or 8; S a multiple of the element
// size): one load, non-temporal when S is SB-aligned, else one unaligned
// (cacheable) access.  Measured on MI355X against reading the two aligned
// 16-byte granules that hold the bytes and funnel-shifting them: the
// 10,000-tensor bfloat16 pack at K = 16 +5.7% (5.21 -> 5.51 TB/s), the
// pipelined step on that group +2.6%.
template <int SB>
__device__ __forceinline__ u4 load_bytes(uintptr_t S) {
    if ((S & (SB - 1)) == 0) {
        if constexpr (SB == 16) return gld_nt<u4>(S);
        const u2 w = gld_nt<u2>(S);
        return u4{w.x, w.y, 0u, 0u};
    }
    if constexpr (SB == 16) return gld_u<u4>(S);
    const u2 w = gld_u<u2>(S);
    return u4{w.x, w.y, 0u, 0u};
}

template <int SB>
__device__ __forceinline__ void store_bytes(uintptr_t D, u4 v) {
    if constexpr (SB == 16) gst_nt<u4>(D, v);
    else gst_nt<u2>(D, u2{v.x, v.y});
}

// Lane l + 1's value in lane l, within a row of 16 lanes (DPP row_shl:1);
// the last lane of a row gets 0.
__device__ __forceinline__ uint32_t from_next_lane(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x101, 0xF, 0xF, true));
}

// Gather of 16-byte windows that consecutive lanes take from consecutive
// addresses (a run of one copy's slots).  A window at an address that is not
// a multiple of 16 spans two aligned granules, the second of which is the
// first granule of the next lane's window.  Each lane loads the granule
// holding its window's start for every window before anything else; it then
// takes the second granule from lane l + 1 when that lane loaded exactly
// that granule (checked on the addresses) and loads it itself otherwise (a
// run's or a row's last lane, the next lane in another run).  N windows per
// lane; window q is skipped when S[q] == 0.  All lanes of the wave must take
// part (the exchange is a cross-lane move).  Measured on MI355X in the
// binary32 tiled pack, with every piece's address found before the first
// load: ResNet-50 at K = 8 6.3-7.1% faster than a search and a load per
// piece in turn.  For 8-byte slots (bfloat16) the same exchange was 3.5%
// slower than two loads per misaligned window; there the addresses-first
// order alone gained 5.6% (10,000 tensors, K = 16).
template <int N>
__device__ __forceinline__ void load_windows(const uintptr_t (&S)[N], u4 (&out)[N]) {
    u4 g0[N], g1[N];
    bool next[N];
#pragma unroll
    for (int q = 0; q < N; ++q) {
        g0[q] = u4{0u, 0u, 0u, 0u};
        if (S[q]) g0[q] = gld_nt<u4>(S[q] & ~uintptr_t(15));
    }
#pragma unroll
    for (int q = 0; q < N; ++q) {
        const uintptr_t g = S[q] & ~uintptr_t(15);
        const uint64_t n = static_cast<uint64_t>(from_next_lane(static_cast<uint32_t>(g))) |
                           (static_cast<uint64_t>(from_next_lane(static_cast<uint32_t>(static_cast<uint64_t>(g) >> 32)))
                            << 32);
        next[q] = S[q] && (S[q] & 15) && n == static_cast<uint64_t>(g) + 16;
        g1[q] = u4{0u, 0u, 0u, 0u};
        if (S[q] && (S[q] & 15) && !next[q]) g1[q] = gld_nt<u4>(g + 16);
    }
#pragma unroll
    for (int q = 0; q < N; ++q) {
        const u4 n4 = u4{from_next_lane(g0[q].x), from_next_lane(g0[q].y), from_next_lane(g0[q].z),
                         from_next_lane(g0[q].w)};
        if (next[q]) g1[q] = n4;
        const uint32_t sh = static_cast<uint32_t>(S[q] & 15);
        out[q] = sh ? funnel(g0[q], g1[q], sh) : g0[q];
    }
}

// Workgroup b moves chunk b of all K copies through LDS, M slots at a time
// (tpack_tile_slots: 1,024 or 2,048 pieces over P, at least 16 slots, at
// most a chunk's), so that both global sides are contiguous:
//   per-copy side  lanes take consecutive slots of one copy (M*SB bytes of
//                  one copy per wave instruction when M >= 64);
//   tensor side    lanes take consecutive pieces in tensor order.
// The tile rows (one per slot, K pieces of SB bytes) are padded by one
// piece so the per-copy phase hits distinct LDS banks.  The chunk's
// segments (tensors) are staged in LDS as chunk-relative starts and, per
// copy, the address of chunk element 0 in that copy's tensor coordinates.
// On the per-copy side a slot inside one tensor moves as one access:
//   pack    one load (unaligned when the slot does not start on a slot
//           boundary; binary32 windows take load_windows);
//   unpack  one store when aligned; else the lane stores the aligned
//           16-byte granule that starts inside its window, assembled from
//           its slot and the copy's next slot, and the first and last slots
//           of a run of whole slots also store the slot itself, unaligned
//           (binary32; an unaligned bfloat16 slot is one unaligned 8-byte
//           store).  Measured on MI355X against element stores for the
//           bytes outside the granules: the 10,000-tensor group's unpack
//           4-6% faster at K = 2-16 (a wave issued every edge store for the
//           whole wave); the pipelined step's scatter, whose tiles end every
//           64 slots, measured 1-3% slower that way and keeps element stores.
// A slot spanning two tensors moves element by element.
// Pieces (one slot of one copy) per LDS tile of the pack and unpack.  The
// binary32 unpack at P >= 16 takes twice as many (measured on MI355X: the
// 10,000-tensor group at K = 16 4.21 -> 4.49 TB/s, ResNet-50 at K = 16 and
// 32 level); pack loses 4-13% with them at every K measured.
#ifndef TC_TPACK_TILE
#define TC_TPACK_TILE 1024
#endif
#ifndef TC_TUNPACK_TILE_WIDE
#define TC_TUNPACK_TILE_WIDE 2048
#endif
#ifndef TC_TPACK_DIRECT
#define TC_TPACK_DIRECT 1
#endif
#ifndef TC_TPACK_GROUP_BYTES
#define TC_TPACK_GROUP_BYTES 128
#endif
#ifndef TC_TPACK_GROUP_WHOLE
#define TC_TPACK_GROUP_WHOLE 1
#endif
// The direct binary32 pack and unpack are compiled for at least 4 waves per
// SIMD (amdgpu_waves_per_eu; they already run at 6, so the hint takes no
// occupancy): measured on MI355X, VGG-16 at K = 4 packs 3% and unpacks 2%
// faster, ResNet-50 at K = 4 4% and 3.5%, whatever the hint's value (4, 5
// or 6).  The same hint on the tiled kernels, the steps and the pipelined
// step measured level or up to 9% slower.
#ifndef TC_TPACK_WAVES_DIRECT
#define TC_TPACK_WAVES_DIRECT 4
#endif


// Longer chunks are taken only while they still give 2,048 workgroups (8 per
// CU): a group of 7,392 elements packed at K = 2 in 2 chunks of 4,096 took
// 5.8 us, in 8 of 1,024 3.8 us.
constexpr int64_t kMinLongerChunks = 2048;

// Slots per LDS tile: the tile's pieces over P, at least 16, and no more
// than the slots of a chunk (TC_TPACK_CHUNK / 4; tiles larger than the chunk
// leave lanes idle), but at least one piece per lane (two for the bfloat16
// pack, whose lanes take two slots), which at P <= 2 sets the size.
template <int P, int ES, bool UNPACK>
constexpr int tpack_tile_slots() {
    constexpr int TILE = UNPACK && ES == 4 && P >= 16 ? TC_TUNPACK_TILE_WIDE : TC_TPACK_TILE;
    constexpr int MT = TILE / P > 16 ? TILE / P : 16;
    constexpr int CS = TC_TPACK_CHUNK / 4;
    constexpr int MIN = (ES == 2 && !UNPACK ? 512 : 256) / P;
    return MT <= CS ? MT : (MIN > CS ? MIN : CS);
}

template <int P, typename T, bool UNPACK, bool DIRECT>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256),
                          amdgpu_waves_per_eu(DIRECT && sizeof(T) == 4 ? TC_TPACK_WAVES_DIRECT : 1)))
void tensor_pack_kernel(TPackArgs a) {
    constexpr int ES = sizeof(T);
    constexpr int SB = 4 * ES;                      // slot bytes
    constexpr int M = tpack_tile_slots<P, ES, UNPACK>();  // slots per LDS tile
    constexpr int ROW = (P + 1) * SB;               // padded tile row, bytes
    __shared__ int32_t s_rel[kMaxStage + 1];
    __shared__ uintptr_t s_base[kMaxStage];
    // one row more than a tile: unpack keeps the next tile's first slot there
    __shared__ __attribute__((aligned(16))) unsigned char s_tile[(M + 1) * ROW];
    // workgroup (chunk, group): copies [kg0, kg0 + K) of chunk, K <= P; the
    // tensor layout's stride is all a.K copies
    const int KS = a.K;
    const int chunk = static_cast<int>(blockIdx.x) / a.groups;
    const int kg0 = (static_cast<int>(blockIdx.x) - chunk * a.groups) * P;
    const int K = KS - kg0 < P ? KS - kg0 : P;
    const int64_t cstart = static_cast<int64_t>(chunk) * a.chunk;
    const int32_t clen = static_cast<int32_t>(a.N - cstart < a.chunk ? a.N - cstart : a.chunk);
    const int32_t lo = a.chunk_first[chunk];
    const int32_t hi = a.chunk_first[chunk + 1];
    const int nseg = hi - lo + 1;
    const int64_t first_start = a.offsets[lo] - cstart;
    const bool rel_staged = nseg <= kMaxStage;
    const bool base_staged = static_cast<int64_t>(nseg) * K <= kMaxStage;
    auto rel_global = [&](int s) -> int32_t { return clamp_rel(a.offsets[lo + s] - cstart, clen); };
    auto base_global = [&](int kk, int s) -> uintptr_t {
        const int64_t st = s == 0 ? first_start : a.offsets[lo + s] - cstart;
        return reinterpret_cast<uintptr_t>(a.ptrs[static_cast<int64_t>(kg0 + kk) * a.n + lo + s]) -
               static_cast<uintptr_t>(st * ES);
    };
    if (rel_staged)
        for (int s = threadIdx.x; s <= nseg; s += 256) s_rel[s] = rel_global(s);
    if (base_staged)
        for (int q = threadIdx.x; q < nseg * K; q += 256) s_base[q] = base_global(q / nseg, q % nseg);
    __syncthreads();
    auto rel = [&](int s) -> int32_t { return rel_staged ? s_rel[s] : rel_global(s); };
    auto base = [&](int kk, int s) -> uintptr_t { return base_staged ? s_base[kk * nseg + s] : base_global(kk, s); };
    auto find = [&](int jr) {  // last segment whose start is <= jr
        int l = 0, h = nseg - 1;
        while (l < h) {
            const int mid = (l + h + 1) >> 1;
            if (rel(mid) <= jr) l = mid; else h = mid - 1;
        }
        return l;
    };
    const uintptr_t tens = reinterpret_cast<uintptr_t>(a.tensor);
    const int64_t slot0 = cstart / 4;
    auto piece = [&](int js, int kk) -> uintptr_t {
        return tens + static_cast<uintptr_t>(((slot0 + js) * KS + kg0 + kk) * SB);
    };
    auto tile = [&](int jl, int kk) -> unsigned char* { return s_tile + jl * ROW + kk * SB; };
    const int nsl = clen / 4;  // whole slots in this chunk
    // a lane's slot is the same in every pass of the unpack's scatter (the
    // binary32 scatter finds its tensor once; for 8-byte slots the extra live
    // registers cost more than the search)
    constexpr bool kSame = SB == 16 && 256 % M == 0;
    if constexpr (DIRECT) {
        // a slot-aligned group and list: lanes take the pieces in tensor order
        // (P per slot, lane i = copy i) and move each slot straight between
        // copy i's tensor and the tensor layout, no tile
        constexpr int SPS = 1024 / P;  // slots per step, four pieces per lane
        const int i = threadIdx.x % P;
        for (int t0 = 0; t0 < nsl; t0 += SPS) {
            u4 v[4];
            uintptr_t dst[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int js = t0 + (threadIdx.x + r * 256) / P;
                if (js >= nsl || i >= K) continue;
                const int jr = 4 * js;
                const uintptr_t per = base(i, find(jr)) + static_cast<uintptr_t>(jr) * ES;
                const uintptr_t tp = piece(js, i);
                v[r] = load_bytes<SB>(UNPACK ? tp : per);
                dst[r] = UNPACK ? per : tp;
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int js = t0 + (threadIdx.x + r * 256) / P;
                if (js >= nsl || i >= K) continue;
                store_bytes<SB>(dst[r], v[r]);
            }
        }
    }
    for (int t0 = 0; !DIRECT && t0 < nsl; t0 += M) {
        const int mt = nsl - t0 < M ? nsl - t0 : M;  // slots in this tile
        // each phase moves M*P = 1024 pieces: 4 per lane, all loads issued
        // before the first write
        constexpr int R = (M * P) / 256;
        if constexpr (!UNPACK) {
            // copies -> tile: lanes walk consecutive slots of one copy
            auto slot_piece = [&](int kk, int js) -> u4 {  // one slot of copy kk
                const int jr = 4 * js;
                int s = find(jr);
                if (jr + 4 <= rel(s + 1)) return load_bytes<SB>(base(kk, s) + static_cast<uintptr_t>(jr) * ES);
                T e4[4];  // the slot spans tensors
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    while (jr + e >= rel(s + 1)) ++s;
                    e4[e] = gld<T>(base(kk, s) + static_cast<uintptr_t>(jr + e) * ES);
                }
                u4 v = u4{0u, 0u, 0u, 0u};
                __builtin_memcpy(&v, e4, SB);
                return v;
            };
            if constexpr (SB == 16) {
                // the addresses of every piece first (the segment searches in
                // LDS), then the loads through load_windows; a slot spanning
                // tensors element by element
                u4 v[R];
                bool ok[R];
                uintptr_t S[R];
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / M, jl = q % M;
                    ok[r] = kk < K && jl < mt;
                    S[r] = 0;
                    if (ok[r]) {
                        const int jr = 4 * (t0 + jl);
                        const int sg = find(jr);
                        if (jr + 4 <= rel(sg + 1)) S[r] = base(kk, sg) + static_cast<uintptr_t>(jr) * ES;
                    }
                }
                load_windows<R>(S, v);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int q = threadIdx.x + r * 256;
                    if (ok[r] && !S[r]) v[r] = slot_piece(q / M, t0 + q % M);
                }
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int q = threadIdx.x + r * 256;
                    if (ok[r]) *reinterpret_cast<u4*>(tile(q % M, q / M)) = v[r];
                }
            } else {
                // 8-byte slots: a lane takes two consecutive slots of one
                // copy, 16 source bytes read with one load when both lie in
                // one tensor; addresses first, then the loads, as above
                constexpr int R2 = R / 2, MH = M / 2;
                u4 v[R2];
                bool ok0[R2], ok1[R2];
                uintptr_t S[R2];
#pragma unroll
                for (int r = 0; r < R2; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / MH, jl = 2 * (q % MH);
                    ok0[r] = kk < K && jl < mt;
                    ok1[r] = kk < K && jl + 1 < mt;
                    S[r] = 0;
                    if (ok1[r]) {
                        const int jr = 4 * (t0 + jl);
                        const int sg = find(jr);
                        if (jr + 8 <= rel(sg + 1)) S[r] = base(kk, sg) + static_cast<uintptr_t>(jr) * ES;
                    }
                }
#pragma unroll
                for (int r = 0; r < R2; ++r)
                    if (S[r]) v[r] = load_bytes<16>(S[r]);
#pragma unroll
                for (int r = 0; r < R2; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / MH, jl = 2 * (q % MH);
                    if (ok0[r] && !S[r]) {
                        const u4 a0 = slot_piece(kk, t0 + jl);
                        const u4 a1 = ok1[r] ? slot_piece(kk, t0 + jl + 1) : u4{0u, 0u, 0u, 0u};
                        v[r] = u4{a0.x, a0.y, a1.x, a1.y};
                    }
                }
#pragma unroll
                for (int r = 0; r < R2; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / MH, jl = 2 * (q % MH);
                    if (ok0[r]) *reinterpret_cast<u2*>(tile(jl, kk)) = u2{v[r].x, v[r].y};
                    if (ok1[r]) *reinterpret_cast<u2*>(tile(jl + 1, kk)) = u2{v[r].z, v[r].w};
                }
            }
            __syncthreads();
            // tile -> tensor, in tensor order
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int q = threadIdx.x + r * 256;
                const int jl = q / P, kk = q % P;
                if (kk >= K || jl >= mt) continue;
                if constexpr (SB == 16) gst_nt<u4>(piece(t0 + jl, kk), *reinterpret_cast<const u4*>(tile(jl, kk)));
                else gst_nt<u2>(piece(t0 + jl, kk), *reinterpret_cast<const u2*>(tile(jl, kk)));
            }
        } else {
            // tensor -> tile, in tensor order.  With a full tile before the
            // chunk's last whole slot, the first K lanes also load the next
            // tile's first slot into the extra row, where the funnel of a
            // misaligned destination's last granule in this tile finds it.
            u4 v[R];
            const bool ahead = SB == 16 && threadIdx.x < K && mt == M && t0 + M < nsl;
            u4 nx = u4{0u, 0u, 0u, 0u};
            if (ahead) nx = gld<u4>(piece(t0 + M, threadIdx.x));
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int q = threadIdx.x + r * 256;
                const int jl = q / P, kk = q % P;
                if (kk >= K || jl >= mt) continue;
                if constexpr (SB == 16) {
                    v[r] = gld_nt<u4>(piece(t0 + jl, kk));
                } else {
                    const u2 w = gld_nt<u2>(piece(t0 + jl, kk));
                    v[r] = u4{w.x, w.y, 0u, 0u};
                }
            }
            if (ahead) *reinterpret_cast<u4*>(tile(M, threadIdx.x)) = nx;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int q = threadIdx.x + r * 256;
                const int jl = q / P, kk = q % P;
                if (kk >= K || jl >= mt) continue;
                if constexpr (SB == 16) *reinterpret_cast<u4*>(tile(jl, kk)) = v[r];
                else *reinterpret_cast<u2*>(tile(jl, kk)) = u2{v[r].x, v[r].y};
            }
            __syncthreads();
            // tile -> copies: lanes walk consecutive slots of one copy (the
            // same slot in every pass when M divides 256)
            const int s_same = kSame && threadIdx.x % M < mt ? find(4 * (t0 + threadIdx.x % M)) : 0;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int q = threadIdx.x + r * 256;
                const int kk = q / M, jl = q % M;
                if (kk >= K || jl >= mt) continue;
                const int js = t0 + jl, jr = 4 * js;
                int s = kSame ? s_same : find(jr);
                const int32_t r1 = rel(s + 1);
                const T* src = reinterpret_cast<const T*>(tile(jl, kk));
                if (jr + 4 <= r1) {
                    const uintptr_t w = base(kk, s) + static_cast<uintptr_t>(jr) * ES;
                    if ((w & (SB - 1)) == 0) {
                        if constexpr (SB == 16) gst_nt<u4>(w, *reinterpret_cast<const u4*>(src));
                        else gst_nt<u2>(w, *reinterpret_cast<const u2*>(src));
                    } else if constexpr (SB == 16) {
                        const uintptr_t G = (w + 15) & ~uintptr_t(15);
                        const uint32_t sh = static_cast<uint32_t>(G - w);  // bytes of this slot before G
                        const int run_lo = (rel(s) + 3) / 4, run_hi = r1 / 4;  // whole slots of this tensor here
                        const bool last = js + 1 >= run_hi;
                        // the run's first and last slots store the slot itself
                        // with one unaligned store (the bytes it shares with a
                        // neighbouring lane's granule get the same values)
                        if (js == run_lo || last) gst_u<u4>(w, *reinterpret_cast<const u4*>(src));
                        if (!last) {
                            // slot js + 1 is a whole slot of the chunk: row jl + 1
                            // of this tile, or the extra row (jl + 1 = mt = M)
                            const u4 next = *reinterpret_cast<const u4*>(tile(jl + 1, kk));
                            gst_nt<u4>(G, funnel(*reinterpret_cast<const u4*>(src), next, sh));
                        }
                    } else {
                        gst_u<u2>(w, *reinterpret_cast<const u2*>(src));
                    }
                } else {  // the slot spans tensors
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        while (jr + e >= rel(s + 1)) ++s;
                        gst<T>(base(kk, s) + static_cast<uintptr_t>(jr + e) * ES, src[e]);
                    }
                }
            }
        }
        __syncthreads();  // the tile is reused
    }
    // the group's last, partial slot: element by element, every copy
    const int rem = clen - 4 * nsl;
    if (threadIdx.x < rem * K) {
        const int kk = threadIdx.x / rem, e = threadIdx.x - kk * rem;
        const int je = 4 * nsl + e;
        int s = find(je);
        while (je >= rel(s + 1)) ++s;
        const uintptr_t t = base(kk, s) + static_cast<uintptr_t>(je) * ES;
        const uintptr_t pc = tens + static_cast<uintptr_t>((((slot0 + nsl) * KS + kg0 + kk) * 4 + e) * ES);
        if (UNPACK) gst<T>(t, gld<T>(pc));
        else gst<T>(pc, gld<T>(t));
    }
}

// ------------------------------------------------------------ pipeline

// The whole step in one pass: pack the K gradient lists into the tensor
// layout, average them, take the fused elastic step, and unpack the K new
// workers into their per-layer tensors.  The same arithmetic as tc_pack_tensor,
// tc_reduce_tensor (AVG), easgd_step_tensor and tc_unpack_tensor in turn, but
// each workgroup takes its chunk of the group through all four with the
// intermediates in LDS and registers: the gradients are read from HBM once
// (not three times) and the new workers are not read back for the unpack.
// This is the on-chip form of pipelining a chunked reduction (Sec. 6.3.2: a
// message split so that its pieces flow through the stages concurrently);
// on one GPU, pipelining across kernel launches loses ~8 us per launch to
// drain and ramp-up and gains nothing from the last-level cache.
//
// Per tile of M slots:
//   gather   lanes walk consecutive slots of one copy's gradient tensors
//            (as tc_pack_tensor) into the LDS tile; the workers and the
//            center of the same slots are loaded in tensor order meanwhile;
//   step     lanes take pieces in tensor order (P lanes per slot, lane i =
//            worker i, as easgd_step_tensor): the packed gradients are
//            written out (optional), the AVG and the center's spread are
//            split butterflies (as tc_reduce_tensor), the workers' new
//            values go to HBM and to the tile;
//   scatter  lanes walk consecutive slots of one copy's parameter tensors
//            (as tc_unpack_tensor); tile edges count as ends of a run of
//            whole slots, so a misaligned destination never needs a slot of
//            the next tile.
struct TPipeArgs {
    const int64_t* offsets;
    const int32_t* chunk_first;
    void* const* gptrs;  // K*n gradient tensors, copy-major
    void* const* xptrs;  // K*n binary32 parameter tensors, copy-major
    void* gt;            // packed gradients, tensor layout, or null
    float* gbar;         // N values: the AVG of the K gradients
    float* x;            // workers, tensor layout
    float* xc;           // N values: the center
    int32_t n, K;
    int64_t N, chunk;
    float eta, rho, a;
};

constexpr int kPipeStage = 512;

// Pieces (one slot of one copy) per step of a workgroup: 256 lanes move
// TILE/256 pieces each.  The straight path (no LDS) holds them in registers;
// the tiled path stages them in LDS, where smaller tiles leave room for more
// workgroups per CU (measured on MI355X: 1024 and 512 best respectively).
// At P >= 16 a tile of 512 pieces holds only 32 slots of each copy, and
// 1024 pieces measure better: the 10,000-tensor bfloat16 group at K = 16
// 4.39 -> 4.56 TB/s, ResNet-50 at K = 16 level or better; 2048 fell to 3.5
// on the 10,000-tensor group, and at P = 8 512 stays best.
#ifndef TC_PIPE_TILE
#define TC_PIPE_TILE 1024
#endif
#ifndef TC_PIPE_TILE_LDS
#define TC_PIPE_TILE_LDS 512
#endif
#ifndef TC_PIPE_TILE_LDS_WIDE
#define TC_PIPE_TILE_LDS_WIDE 1024
#endif
// At P = 32 (K = 17 to 32) tiles of 512 pieces, 16 slots, measured better
// than 1,024 on the ResNet-50 group: K = 17 +4%, K = 20 +5%, K = 32 +4.4%,
// bfloat16 gradients at K = 17 +1.5%; 2,048 lost 11-34%.  (At P = 64 both
// give the 16-slot minimum; at P = 16, 512 lost 1.5% at K = 16.)
#ifndef TC_PIPE_TILE_LDS_P32
#define TC_PIPE_TILE_LDS_P32 512
#endif


__device__ __forceinline__ f4 widen_piece(u4 v, int es) {
    if (es == 4) return f4{__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w)};
    return f4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
              __uint_as_float(v.y & 0xffff0000u)};
}

__device__ __forceinline__ float comp(f4 v, int c) { return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w; }

template <int P, typename T, bool WG, typename I, bool DIRECT>
__global__ __launch_bounds__(256) void tensor_pipeline_kernel(TPipeArgs a) {
    constexpr int ES = sizeof(T);
    constexpr int SB = 4 * ES;                         // gradient slot bytes
    constexpr int TILE = DIRECT ? TC_PIPE_TILE : P == 32 ? TC_PIPE_TILE_LDS_P32 : P >= 16 ? TC_PIPE_TILE_LDS_WIDE : TC_PIPE_TILE_LDS;
    constexpr int M = TILE / P > 16 ? TILE / P : 16;  // slots per tile
    constexpr int R = (M * P) / 256;                                 // pieces per lane and phase
    constexpr int ROWG = (P + 1) * SB, ROWX = (P + 1) * 16;
    __shared__ int32_t s_rel[kPipeStage + 1];
    __shared__ uintptr_t s_gbase[kPipeStage];
    __shared__ uintptr_t s_xbase[kPipeStage];
    __shared__ __attribute__((aligned(16))) unsigned char s_tile[M * ROWX];
    const int K = a.K;
    const int i = threadIdx.x % P;
    const int64_t cstart = static_cast<int64_t>(blockIdx.x) * a.chunk;
    const int32_t clen = static_cast<int32_t>(a.N - cstart < a.chunk ? a.N - cstart : a.chunk);
    const int32_t lo = a.chunk_first[blockIdx.x];
    const int32_t hi = a.chunk_first[blockIdx.x + 1];
    const int nseg = hi - lo + 1;
    const bool rel_staged = nseg <= kPipeStage;
    const bool base_staged = static_cast<int64_t>(nseg) * K <= kPipeStage;
    auto rel_global = [&](int s) -> int32_t { return clamp_rel(a.offsets[lo + s] - cstart, clen); };
    auto base_global = [&](void* const* ptrs, int es, int kk, int s) -> uintptr_t {
        return reinterpret_cast<uintptr_t>(ptrs[static_cast<int64_t>(kk) * a.n + lo + s]) -
               static_cast<uintptr_t>((a.offsets[lo + s] - cstart) * es);
    };
    const int nsl = clen / 4;  // whole slots in this chunk
    if (rel_staged)
        for (int s = threadIdx.x; s <= nseg; s += 256) s_rel[s] = rel_global(s);
    if (base_staged)
        for (int q = threadIdx.x; q < nseg * K; q += 256) {
            s_gbase[q] = base_global(a.gptrs, ES, q / nseg, q % nseg);
            s_xbase[q] = base_global(a.xptrs, 4, q / nseg, q % nseg);
        }
    __syncthreads();
    auto rel = [&](int s) -> int32_t { return rel_staged ? s_rel[s] : rel_global(s); };
    auto gbase = [&](int kk, int s) -> uintptr_t {
        return base_staged ? s_gbase[kk * nseg + s] : base_global(a.gptrs, ES, kk, s);
    };
    auto xbase = [&](int kk, int s) -> uintptr_t {
        return base_staged ? s_xbase[kk * nseg + s] : base_global(a.xptrs, 4, kk, s);
    };
    auto find = [&](int jr) {  // last segment whose start is <= jr
        int l = 0, h = nseg - 1;
        while (l < h) {
            const int mid = (l + h + 1) >> 1;
            if (rel(mid) <= jr) l = mid; else h = mid - 1;
        }
        return l;
    };
    auto gtile = [&](int jl, int kk) -> unsigned char* { return s_tile + jl * ROWG + kk * SB; };
    auto xtile = [&](int jl, int kk) -> unsigned char* { return s_tile + jl * ROWX + kk * 16; };
    const int64_t slot0 = cstart / 4;
    const f4 rho = f4(a.rho), neg_eta = f4(-a.eta), alpha = f4(a.a);
    // The step on one piece (slot J of worker i): the packed gradient out,
    // the AVG and the center from the split butterflies, the new worker out
    // and returned.  Every lane calls it (the butterflies need all lanes).
    auto step = [&](I J, bool slot, bool live, u4 raw, f4 x, f4 c) -> f4 {
        if constexpr (WG)
            if (live) store_bytes<SB>(reinterpret_cast<uintptr_t>(a.gt) + (J * I(K) + I(i)) * I(SB), raw);
        const f4 g = widen_piece(raw, ES);
        const f4 d = live ? x - c : f4(0.0f);
        const f4 xn = fma4(neg_eta, fma4(rho, d, g), x);
        if constexpr (P >= 4) {
            // lanes 0-3 of the slot's group hold one component each
            const float gs = div_k<P>(split_group_sum<P>(g, threadIdx.x), K);
            const float ds = split_group_sum<P>(d, threadIdx.x);
            const int cp = comp_of_lane(i);
            if (slot && i < 4) {
                __builtin_nontemporal_store(gs, a.gbar + (J * I(4) + I(cp)));
                __builtin_nontemporal_store(__builtin_fmaf(a.a, ds, comp(c, cp)), a.xc + (J * I(4) + I(cp)));
            }
        } else {
            const f4 gs = div_k<P>(group_sum4<P>(g), K);
            const f4 cn = fma4(alpha, group_sum4<P>(d), c);
            if (slot && i == 0) {
                store_slot(a.gbar, J, gs);
                store_slot(a.xc, J, cn);
            }
        }
        if (live) store_slot(a.x, J * I(K) + I(i), xn);
        return xn;
    };
    if constexpr (DIRECT) {
        // every whole slot lies inside one tensor and every tensor is
        // slot-aligned in every copy: the chunk moves straight between
        // registers and the per-layer tensors, without the tiles
        for (int t0 = 0; t0 < nsl; t0 += M) {
            const int mt = nsl - t0 < M ? nsl - t0 : M;
            f4 xv[R], cv[R];
            u4 gr[R];
            int seg[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int jl = (threadIdx.x + r * 256) / P;
                const I J = static_cast<I>(slot0 + t0 + jl);
                const bool live = jl < mt && i < K;
                cv[r] = jl < mt ? load_slot(a.xc, J) : f4(0.0f);
                xv[r] = live ? load_slot(a.x, J * I(K) + I(i)) : f4(0.0f);
                gr[r] = u4{0u, 0u, 0u, 0u};
                seg[r] = 0;
                if (live) {
                    const int jr = 4 * (t0 + jl);
                    seg[r] = find(jr);
                    gr[r] = load_bytes<SB>(gbase(i, seg[r]) + static_cast<uintptr_t>(jr) * ES);
                }
            }
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int jl = (threadIdx.x + r * 256) / P;
                const I J = static_cast<I>(slot0 + t0 + jl);
                const bool live = jl < mt && i < K;
                const f4 xn = step(J, jl < mt, live, gr[r], xv[r], cv[r]);
                if (live) gst_nt<u4>(xbase(i, seg[r]) + static_cast<uintptr_t>(4 * (t0 + jl)) * 4, __builtin_bit_cast(u4, xn));
            }
        }
    }
    for (int t0 = 0; !DIRECT && t0 < nsl; t0 += M) {
        const int mt = nsl - t0 < M ? nsl - t0 : M;
        // gather: gradients into the tile; workers and center in registers
        {
            auto slot_piece = [&](int kk, int js) -> u4 {  // one slot of copy kk
                const int jr = 4 * js;
                int s = find(jr);
                if (jr + 4 <= rel(s + 1)) return load_bytes<SB>(gbase(kk, s) + static_cast<uintptr_t>(jr) * ES);
                T e4[4];  // the slot spans tensors
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    while (jr + e >= rel(s + 1)) ++s;
                    e4[e] = gld<T>(gbase(kk, s) + static_cast<uintptr_t>(jr + e) * ES);
                }
                u4 v = u4{0u, 0u, 0u, 0u};
                __builtin_memcpy(&v, e4, SB);
                return v;
            };
            if constexpr (SB == 16) {
                // as in tc_pack_tensor: addresses first, then load_windows
                u4 v[R];
                bool ok[R];
                uintptr_t S[R];
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / M, jl = q % M;
                    ok[r] = kk < K && jl < mt;
                    S[r] = 0;
                    if (ok[r]) {
                        const int jr = 4 * (t0 + jl);
                        const int sg = find(jr);
                        if (jr + 4 <= rel(sg + 1)) S[r] = gbase(kk, sg) + static_cast<uintptr_t>(jr) * ES;
                    }
                }
                load_windows<R>(S, v);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int q = threadIdx.x + r * 256;
                    if (ok[r] && !S[r]) v[r] = slot_piece(q / M, t0 + q % M);
                }
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int q = threadIdx.x + r * 256;
                    if (ok[r]) *reinterpret_cast<u4*>(gtile(q % M, q / M)) = v[r];
                }
            } else {
                // 8-byte slots: two consecutive slots of one copy per lane,
                // as in tc_pack_tensor
                constexpr int R2 = R / 2, MH = M / 2;
                u4 v[R2];
                bool ok0[R2], ok1[R2];
                uintptr_t S[R2];
#pragma unroll
                for (int r = 0; r < R2; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / MH, jl = 2 * (q % MH);
                    ok0[r] = kk < K && jl < mt;
                    ok1[r] = kk < K && jl + 1 < mt;
                    S[r] = 0;
                    if (ok1[r]) {
                        const int jr = 4 * (t0 + jl);
                        const int sg = find(jr);
                        if (jr + 8 <= rel(sg + 1)) S[r] = gbase(kk, sg) + static_cast<uintptr_t>(jr) * ES;
                    }
                }
#pragma unroll
                for (int r = 0; r < R2; ++r)
                    if (S[r]) v[r] = load_bytes<16>(S[r]);
#pragma unroll
                for (int r = 0; r < R2; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / MH, jl = 2 * (q % MH);
                    if (ok0[r] && !S[r]) {
                        const u4 a0 = slot_piece(kk, t0 + jl);
                        const u4 a1 = ok1[r] ? slot_piece(kk, t0 + jl + 1) : u4{0u, 0u, 0u, 0u};
                        v[r] = u4{a0.x, a0.y, a1.x, a1.y};
                    }
                }
#pragma unroll
                for (int r = 0; r < R2; ++r) {
                    const int q = threadIdx.x + r * 256;
                    const int kk = q / MH, jl = 2 * (q % MH);
                    if (ok0[r]) *reinterpret_cast<u2*>(gtile(jl, kk)) = u2{v[r].x, v[r].y};
                    if (ok1[r]) *reinterpret_cast<u2*>(gtile(jl + 1, kk)) = u2{v[r].z, v[r].w};
                }
            }
        }
        f4 xv[R], cv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int jl = (threadIdx.x + r * 256) / P;
            const I J = static_cast<I>(slot0 + t0 + jl);
            cv[r] = jl < mt ? load_slot(a.xc, J) : f4(0.0f);
            xv[r] = jl < mt && i < K ? load_slot(a.x, J * I(K) + I(i)) : f4(0.0f);
        }
        __syncthreads();
        // step, in tensor order
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int jl = (threadIdx.x + r * 256) / P;
            const I J = static_cast<I>(slot0 + t0 + jl);
            const bool slot = jl < mt, live = slot && i < K;
            u4 raw = u4{0u, 0u, 0u, 0u};
            if (live) {
                if constexpr (SB == 16) raw = *reinterpret_cast<const u4*>(gtile(jl, i));
                else {
                    const u2 w = *reinterpret_cast<const u2*>(gtile(jl, i));
                    raw = u4{w.x, w.y, 0u, 0u};
                }
            }
            xv[r] = step(J, slot, live, raw, xv[r], cv[r]);
        }
        if constexpr (ROWG != ROWX) __syncthreads();  // the gradient pieces are read
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int jl = (threadIdx.x + r * 256) / P;
            if (jl < mt && i < K) *reinterpret_cast<f4*>(xtile(jl, i)) = xv[r];
        }
        __syncthreads();
        // scatter: lanes walk consecutive slots of one copy's parameters
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int q = threadIdx.x + r * 256;
            const int kk = q / M, jl = q % M;
            if (kk >= K || jl >= mt) continue;
            const int js = t0 + jl, jr = 4 * js;
            int s = find(jr);
            const int32_t r1 = rel(s + 1);
            const float* src = reinterpret_cast<const float*>(xtile(jl, kk));
            if (jr + 4 <= r1) {
                const uintptr_t w = xbase(kk, s) + static_cast<uintptr_t>(jr) * 4;
                if ((w & 15) == 0) {
                    gst_nt<u4>(w, *reinterpret_cast<const u4*>(src));
                } else {
                    // whole slots of this tensor in this tile: [run_lo, run_hi)
                    const int rl = (rel(s) + 3) / 4, rh = r1 / 4;
                    const int run_lo = rl > t0 ? rl : t0, run_hi = rh < t0 + mt ? rh : t0 + mt;
                    const uintptr_t G = (w + 15) & ~uintptr_t(15);
                    const uint32_t sh = static_cast<uint32_t>(G - w);  // bytes of this slot before G
                    if (js == run_lo)  // bytes before the first granule
                        for (uint32_t e = 0; e < sh / 4; ++e) gst<float>(w + e * 4, src[e]);
                    if (js + 1 < run_hi) {
                        const u4 next = *reinterpret_cast<const u4*>(xtile(jl + 1, kk));
                        gst_nt<u4>(G, funnel(*reinterpret_cast<const u4*>(src), next, sh));
                    } else {  // the run's last slot: bytes after G
                        for (uint32_t e = sh / 4; e < 4; ++e) gst<float>(w + e * 4, src[e]);
                    }
                }
            } else {  // the slot spans tensors
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    while (jr + e >= rel(s + 1)) ++s;
                    gst<float>(xbase(kk, s) + static_cast<uintptr_t>(jr + e) * 4, src[e]);
                }
            }
        }
        __syncthreads();  // the tile is reused
    }
}

// The group's last, partial slot (N not a multiple of 4) in a launch of its
// own, one lane per element and all K copies in it, with the arithmetic and
// summation order of the main kernel (kept apart so that the main kernel's
// registers are not sized for it).
template <int P, typename T, bool WG>
__global__ __launch_bounds__(64) void tensor_pipeline_tail_kernel(TPipeArgs a) {
    constexpr int ES = sizeof(T);
    const int64_t nsl = a.N / 4;  // whole slots of the group
    const int e = threadIdx.x;
    const int64_t je = 4 * nsl + e;
    if (je >= a.N) return;
    int l = 0, h = a.n - 1;  // the last tensor whose start is <= je
    while (l < h) {
        const int mid = (l + h + 1) >> 1;
        if (a.offsets[mid] <= je) l = mid; else h = mid - 1;
    }
    const int64_t loc = je - a.offsets[l];
    const int K = a.K;
    const float c = a.xc[je];
    float gv[P], dv[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
        gv[q] = 0.0f;
        dv[q] = 0.0f;
        if (q >= K) continue;
        const int64_t tq = static_cast<int64_t>(q) * a.n + l;
        const T graw = gld<T>(reinterpret_cast<uintptr_t>(a.gptrs[tq]) + static_cast<uintptr_t>(loc) * ES);
        const int64_t idx = (nsl * K + q) * 4 + e;
        if constexpr (WG) gst<T>(reinterpret_cast<uintptr_t>(a.gt) + static_cast<uintptr_t>(idx) * ES, graw);
        gv[q] = ES == 4 ? __uint_as_float(static_cast<uint32_t>(graw)) : bf16_to_f32(static_cast<uint16_t>(graw));
        const float xo = a.x[idx];
        dv[q] = xo - c;
        const float xn = __builtin_fmaf(-a.eta, __builtin_fmaf(a.rho, dv[q], gv[q]), xo);
        a.x[idx] = xn;
        gst<float>(reinterpret_cast<uintptr_t>(a.xptrs[tq]) + static_cast<uintptr_t>(loc) * 4, xn);
    }
    a.gbar[je] = div_k<P>(Tree<P>::sum(gv), K);
    a.xc[je] = __builtin_fmaf(a.a, Tree<P>::sum(dv), c);
}

// ---------------------------------------------------------- launching

// Slots per lane: enough that a wave's single-stream output covers a
// 128-byte line (P/8 for P >= 16); the reduction takes at least 2, the
// step 1 (measured), and the step at most 4 (8 at P = 64 needed all 256
// VGPRs, one wave per SIMD).
// bfloat16 inputs read one copy per lane (odd K; 8-byte slots) take four
// times the slots, at most 16 (measured at K = 16: 4.6 TB/s with twice, 4.9
// with four times, 3.9 with eight times the binary32 count).
constexpr int treduce_unroll(int P, int es) {
    const int u = P / 8 > 2 ? P / 8 : 2;
    return es == 2 ? (4 * u < 16 ? 4 * u : 16) : u;
}
// bfloat16 pairs (even K; 16 bytes per lane, L = P / 2 lanes per slot):
// the binary32 count for L lanes, times TC_TREDUCE_PAIR_SCALE, at most 16
// (measured at K = 16: 6.27-6.34 TB/s once, 6.35-6.40 twice, 6.21-6.26
// four times); at L <= 2 (K = 2, 4) two slots, where four measured 3-7%
// slower on ResNet-50, VGG-16 and 10,000 small tensors, and one within 3%.
#ifndef TC_TREDUCE_PAIR_SCALE
#define TC_TREDUCE_PAIR_SCALE 2
#endif
#ifndef TC_TREDUCE_PAIR
#define TC_TREDUCE_PAIR 1
#endif
constexpr int treduce_pair_unroll(int L) {
    if (L <= 2) return 2;
    const int u = TC_TREDUCE_PAIR_SCALE * (L / 8 > 2 ? L / 8 : 2);
    return u < 16 ? u : 16;
}
constexpr int teasgd_unroll(int P) { return P >= 32 ? 4 : P / 8 > 1 ? P / 8 : 1; }

template <int P, typename T, bool PAIR>
hipError_t run_treduce_as(int K, const void* in, float* out, int op, int64_t n, hipStream_t s) {
    constexpr int L = PAIR ? P / 2 : P;
    constexpr int U = PAIR ? treduce_pair_unroll(L) : treduce_unroll(P, sizeof(T));
    constexpr int SPB = 256 / L;
    TReduceArgs<T> a{static_cast<const T*>(in), out, n / 4, n, K, op};
    const int64_t blocks = (a.nslot + SPB * U - 1) / (SPB * U);
    dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
    if ((a.nslot + 1) * K * 16 < (int64_t(1) << 32))
        hipLaunchKernelGGL((tensor_reduce_kernel<P, T, U, uint32_t, PAIR>), grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((tensor_reduce_kernel<P, T, U, int64_t, PAIR>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int P, typename T>
hipError_t run_treduce(int K, const void* in, float* out, int op, int64_t n, hipStream_t s) {
    if constexpr (sizeof(T) == 2 && P >= TC_TRD_STAGED_MINP) {
        if (TC_TRD_STAGED && K != P) {
            // as many slots as fill R rounds of the 256 lanes (P / 2 < K < P),
            // rounded down to even
            constexpr int R = TC_TRD_STAGED_R;
            const int S = (256 * R / K) & ~1;
            TReduceArgs<T> a{static_cast<const T*>(in), out, n / 4, n, K, op};
            const int64_t blocks = (a.nslot + S - 1) / S;
            dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
            constexpr bool PAIR = true;  // two copies a lane
            if ((a.nslot + 1) * K * 16 < (int64_t(1) << 32))
                hipLaunchKernelGGL((tensor_reduce_staged_kernel<P, T, R, uint32_t, PAIR>), grid, dim3(256), 0, s, a, S);
            else
                hipLaunchKernelGGL((tensor_reduce_staged_kernel<P, T, R, int64_t, PAIR>), grid, dim3(256), 0, s, a, S);
            return hipGetLastError();
        }
    }
    if constexpr (sizeof(T) == 2 && P >= 2)
        if (TC_TREDUCE_PAIR && K % 2 == 0) return run_treduce_as<P, T, true>(K, in, out, op, n, s);
    return run_treduce_as<P, T, false>(K, in, out, op, n, s);
}

template <int P, typename T, bool RED>
hipError_t run_teasgd_as(const TEasgdArgs<T>& a, hipStream_t s) {
    if constexpr (P >= TC_TEA_STAGED_MINP) {
        if (a.K != P) {
            // binary32 gradients: R slot groups' worth of slots, whose pieces
            // fill K / P of the R rounds; bfloat16: as many as fill them
            // (P / 2 < K < P).  Measured on MI355X, ResNet-50 group, against
            // the slot mapping: binary32 step +2-11%, with the reduction
            // -1 to +14% (K = 17 to 48); filling the rounds lost 3-5 points
            // of that.  bfloat16 step -1 to +14%, with the reduction +6 to
            // +30%, where R slot groups had gained up to 14.
            constexpr int R = TC_TEA_STAGED_R;
            const int S = sizeof(T) == 4 ? R * (256 / P) : 256 * R / a.K;
            const int64_t blocks = (a.nslot + S - 1) / S;
            dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
            if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
                hipLaunchKernelGGL((tensor_easgd_staged_kernel<P, T, R, uint32_t, RED>), grid, dim3(256), 0, s, a, S);
            else
                hipLaunchKernelGGL((tensor_easgd_staged_kernel<P, T, R, int64_t, RED>), grid, dim3(256), 0, s, a, S);
            return hipGetLastError();
        }
    }
    constexpr int U = teasgd_unroll(P);
    constexpr int SPB = 256 / P;
    const int64_t blocks = (a.nslot + SPB * U - 1) / (SPB * U);
    dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
    if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
        hipLaunchKernelGGL((tensor_easgd_kernel<P, T, U, uint32_t, RED>), grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((tensor_easgd_kernel<P, T, U, int64_t, RED>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int P, typename T>
hipError_t run_teasgd(int K, float* x, const void* g, float* xc, float* out, int op, float eta, float rho, int64_t n,
                      hipStream_t s) {
    TEasgdArgs<T> a{x, static_cast<const T*>(g), xc, n / 4, n, eta, rho, eta * rho, K, out, op};
    return out ? run_teasgd_as<P, T, true>(a, s) : run_teasgd_as<P, T, false>(a, s);
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
hipError_t dispatch_teasgd(int K, float* x, const void* g, float* xc, float* out, int op, float eta, float rho,
                           int64_t n, hipStream_t s) {
    switch (next_pow2(K)) {
#define TC_CASE(p) \
    case p: return run_teasgd<p, T>(K, x, g, xc, out, op, eta, rho, n, s);
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

hipError_t launch_tensor_easgd(int K, float* x, const void* g, int g_dtype, float* xc, float* out, int op, float eta,
                               float rho, int64_t n, hipStream_t stream) {
    if (g_dtype == TC_BF16) return dispatch_teasgd<uint16_t>(K, x, g, xc, out, op, eta, rho, n, stream);
    return dispatch_teasgd<float>(K, x, g, xc, out, op, eta, rho, n, stream);
}

#ifndef TC_TPACK_FINE_K
#define TC_TPACK_FINE_K 12
#endif
template <int P, bool DIRECT>
hipError_t run_tpack(const tc_tensorlist* tl, void* tensor, bool unpack, hipStream_t stream) {
    const tc_group* g = tl->g;
    // Chunks:
    // - at P <= 2 a chunk of TC_TPACK_CHUNK elements moves little (4-16 KB),
    //   so these lists take the longer chunks of the separate-buffer pack
    //   (2,048 or 4,096 elements; measured on MI355X, K = 1 and 2 on
    //   ResNet-50, VGG-16 and 10,000 small tensors: pack 2-80% faster,
    //   unpack 12-57% in bfloat16 and 20-35% for misaligned lists), except
    //   the direct binary32 unpack at P = 2 (1-3% slower with them), and
    //   groups too small to fill the chip with them (kMinLongerChunks);
    // - through the tiles, where a tile fits in its chunks (P >= 8; at P = 4
    //   the tiles would leave half the lanes idle), the shorter chunking
    //   (TC_TPACK_CHUNK_FINE) serves unpack on a group of large tensors or
    //   with the copies taken in groups, and pack from K = TC_TPACK_FINE_K.
    //   Measured on MI355X against TC_TPACK_CHUNK: pack +2.5-5.5% at K = 12
    //   to 31 on ResNet-50 (3-6.6% slower at K = 9), +3% on the 10,000-tensor
    //   group at K = 16; its binary32 unpack +5% at K = 16 (copy groups) but
    //   6.5% slower at K = 12 (no groups).
    constexpr int fine_slots = TC_TPACK_CHUNK_FINE / 4;
    const int tile = unpack ? (tl->elem == 2 ? tpack_tile_slots<P, 2, true>() : tpack_tile_slots<P, 4, true>())
                            : (tl->elem == 2 ? tpack_tile_slots<P, 2, false>() : tpack_tile_slots<P, 4, false>());
    const bool fits = tile <= fine_slots;
    const bool longer =
        P <= 2 && !(DIRECT && unpack && tl->elem == 4 && P == 2) && g->sep.nchunks >= kMinLongerChunks;
    const bool grouped = P < next_pow2(tl->K);
    const bool fine = !DIRECT && fits && (unpack ? g->large || grouped : tl->K >= TC_TPACK_FINE_K);
    const tc_chunking& c = longer ? g->sep : fine ? g->tpack_fine : g->tpack;
    const int groups = (tl->K + P - 1) / P;
    TPackArgs a{g->d_offsets, c.d_first, tl->d_ptrs, tensor, g->n, tl->K, g->N, c.chunk, groups};
    dim3 grid(static_cast<unsigned>(c.nchunks * groups));
    if (tl->elem == 2) {
        if (unpack) hipLaunchKernelGGL((tensor_pack_kernel<P, uint16_t, true, DIRECT>), grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((tensor_pack_kernel<P, uint16_t, false, DIRECT>), grid, dim3(256), 0, stream, a);
    } else {
        if (unpack) hipLaunchKernelGGL((tensor_pack_kernel<P, uint32_t, true, DIRECT>), grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((tensor_pack_kernel<P, uint32_t, false, DIRECT>), grid, dim3(256), 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_tensor_pack(const tc_tensorlist* tl, void* tensor, bool unpack, hipStream_t stream) {
    const tc_group* g = tl->g;
    // straight through registers when every tensor boundary before the last,
    // partial slot falls on a slot boundary, every tensor of the list is
    // slot-aligned and a wave still moves >= 256 contiguous bytes of each copy
    // ((64 / P) slots of 4 * elem bytes: P <= 4 for binary32, P <= 2 for
    // bfloat16).  Measured on MI355X: VGG-16 at K = 4 packs 5% faster that way
    // in binary32, while at K = 8 (128 bytes per copy and wave) the tiles' 2 KB
    // runs win; in bfloat16 the tiles win at K = 4 (128 bytes per copy and
    // wave; VGG-16 +15%, ResNet-50 +17%) and lose at K = 2 (up to 19%).
    const bool direct = TC_TPACK_DIRECT && (64 / next_pow2(tl->K)) * 4 * tl->elem >= 256 && g->slot_bounds &&
                        tl->slot_aligned;
    // Through the tiles at P = 16 and 32, the copies are taken in groups whose
    // part of a slot row is TC_TPACK_GROUP_BYTES (one 128-byte line: 8
    // binary32 or 16 bfloat16 copies), each group by a workgroup of its own,
    // whose tile, registers and per-copy side are those of P = 8 (or 16).
    // Measured on MI355X against one workgroup for all K copies: the
    // 10,000-tensor group's binary32 unpack +12% at K = 16 and +6.5% at
    // K = 32 (its bfloat16 pack +2% at K = 32), ResNet-50 and VGG-16 at K =
    // 16 and 32 level to +3%; at K = 64 up to 4% slower, and groups of 64
    // bytes (half lines) 11-33% slower everywhere.  Only when the groups are
    // whole (TC_TPACK_GROUP_WHOLE: K a multiple of the group size): a last,
    // partial group writes pieces of every slot row that fill no line, and
    // leaves most of its lanes idle.  With it, ResNet-50 at K = 9 to 15 and
    // 31 packed at 2.0-2.2 TB/s; in one group, 5.3-5.9 (unpack +20-38%).
    const int pg = TC_TPACK_GROUP_BYTES / (4 * tl->elem);
    const int pk = next_pow2(tl->K);
    const int pt = !direct && pg > 0 && pk > pg && pk <= 32 && (!TC_TPACK_GROUP_WHOLE || tl->K % pg == 0) ? pg : pk;
    switch (pt) {
#define TC_CASE(p) \
    case p: return direct ? run_tpack<p, true>(tl, tensor, unpack, stream) \
                          : run_tpack<p, false>(tl, tensor, unpack, stream);
        TC_FOR_P(TC_CASE)
#undef TC_CASE
        default: return hipErrorInvalidValue;
    }
}

template <int P, typename T, bool DIRECT>
hipError_t run_tpipe(const TPipeArgs& a, unsigned blocks, hipStream_t stream) {
    dim3 grid(blocks);
    const int64_t nslot = a.N / 4;
    if ((nslot + 1) * a.K * 16 < (int64_t(1) << 32)) {
        if (a.gt) hipLaunchKernelGGL((tensor_pipeline_kernel<P, T, true, uint32_t, DIRECT>), grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((tensor_pipeline_kernel<P, T, false, uint32_t, DIRECT>), grid, dim3(256), 0, stream, a);
    } else {
        if (a.gt) hipLaunchKernelGGL((tensor_pipeline_kernel<P, T, true, int64_t, DIRECT>), grid, dim3(256), 0, stream, a);
        else hipLaunchKernelGGL((tensor_pipeline_kernel<P, T, false, int64_t, DIRECT>), grid, dim3(256), 0, stream, a);
    }
    return hipGetLastError();
}

// The straight path pays only while a wave moves at least 128 contiguous
// bytes of every copy's gradient tensors: (64 / P) slots of 4 elements.
// Measured on ResNet-50 and VGG-16 groups: at P = 16 binary32 it ran at 3.9
// against 5.0 TB/s tiled, at P = 8 bfloat16 at 5.0 against 5.2, and 3 to 7
// times slower at P = 32 and 64; within the bound it is 3-7% ahead.
template <int P, typename T>
constexpr bool pipe_direct_pays() { return (64 / P) * 4 * static_cast<int>(sizeof(T)) >= 128; }

// At P <= 2 a step's tile holds 256 to 1,024 slots while a 512-element
// chunk holds 128, so most of a lane's pieces fall past the chunk's end;
// those lists take the tensor-layout pack's 1,024-element chunks instead,
// except binary32 gradients on the straight path at P = 2.  Measured on
// MI355X against the 512-element chunks: K = 1 32-55% faster (ResNet-50,
// 10,000 tensors), K = 2 with bfloat16 gradients or misaligned lists 14-26%
// faster; the straight binary32 path at K = 2 6% faster on ResNet-50 but 9%
// slower on VGG-16; at P = 4 the longer chunks lost 4-8%, and the separate-
// buffer pack's chunks (2,048 or 4,096 elements) gained less at P <= 2.
// On groups of large tensors from K = TC_PIPE_FINE_K, chunks of
// TC_PIPE_CHUNK_FINE elements: each workgroup then moves half the bytes, and
// those resident at one time cover a smaller window of the buffers.
// Measured on MI355X against 512 elements: ResNet-50 K = 8 +2.5%, K = 16 to
// 64 +1.3-2.6%, VGG-16 K = 8 and 16 +2-3%, bfloat16 gradients at K = 8 and
// 16 +5.7-7.3%; at K = 5 2% slower, and on the 10,000-tensor group 3-4%
// slower at K = 16.
#ifndef TC_PIPE_FINE_K
#define TC_PIPE_FINE_K 8
#endif
template <int P, typename T>
hipError_t run_tpipe(const tc_group* g, TPipeArgs a, bool direct, hipStream_t stream) {
    const bool longer = (P == 1 || (P == 2 && !(direct && sizeof(T) == 4))) && g->tpack.nchunks >= kMinLongerChunks;
    const bool fine = !longer && TC_PIPE_FINE_K > 0 && g->large && a.K >= TC_PIPE_FINE_K;
    const tc_chunking& c = longer ? g->tpack : fine ? g->pipe_fine : g->pipe;
    a.chunk_first = c.d_first;
    a.chunk = c.chunk;
    const unsigned blocks = static_cast<unsigned>(c.nchunks);
    hipError_t e;
    if constexpr (pipe_direct_pays<P, T>())
        e = direct ? run_tpipe<P, T, true>(a, blocks, stream) : run_tpipe<P, T, false>(a, blocks, stream);
    else
        e = run_tpipe<P, T, false>(a, blocks, stream);
    if (e != hipSuccess || a.N % 4 == 0) return e;
    if (a.gt) hipLaunchKernelGGL((tensor_pipeline_tail_kernel<P, T, true>), dim3(1), dim3(64), 0, stream, a);
    else hipLaunchKernelGGL((tensor_pipeline_tail_kernel<P, T, false>), dim3(1), dim3(64), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_tensor_pipeline(const tc_tensorlist* grads, const tc_tensorlist* params, void* gt, float* gbar,
                                  float* x, float* xc, float eta, float rho, hipStream_t stream) {
    const tc_group* g = grads->g;
    TPipeArgs a{g->d_offsets, g->pipe.d_first, grads->d_ptrs, params->d_ptrs, gt, gbar, x, xc,
                g->n, grads->K, g->N, g->pipe.chunk, eta, rho, eta * rho};
    const bool bf16 = grads->elem == 2;
    // straight between registers and the per-layer tensors when every tensor
    // boundary before the last, partial slot falls on a slot boundary and
    // every tensor of both lists is slot-aligned (and K is small enough,
    // pipe_direct_pays)
    const bool direct = g->slot_bounds && grads->slot_aligned && params->slot_aligned;
    switch (next_pow2(grads->K)) {
#define TC_CASE(p) \
    case p: return bf16 ? run_tpipe<p, uint16_t>(g, a, direct, stream) : run_tpipe<p, uint32_t>(g, a, direct, stream);
        TC_FOR_P(TC_CASE)
#undef TC_CASE
        default: return hipErrorInvalidValue;
    }
}

#ifndef TC_TASYNC_U
#define TC_TASYNC_U 2
#endif
// Plain SGD on the tensor layout is elementwise over the whole buffer: when K
// is not a power of two, lanes take its pieces one after another (as the
// dense broadcast does), so no lane of a slot group idles.  The arithmetic
// per piece is the slot kernel's.
template <typename T, typename I>
__global__ __launch_bounds__(256) void tensor_sgd_dense_kernel(TStepArgs<T> a) {
    const I np = static_cast<I>(a.nslot) * static_cast<I>(a.K);
    const I p = static_cast<I>(tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x)) * I(256) + threadIdx.x;
    if (p < np) {
        const f4 x = load_slot(a.x, p), g = load_slot(static_cast<const T*>(a.g), p);
        store_slot(a.x, p, fma4(f4(-a.s0), g, x));
    }
    if (blockIdx.x == gridDim.x - 1) tensor_step_tail<TOp::Sgd, 1, T>(a);  // P is not used by plain SGD
}

// Synchronous SGD staged through LDS (P >= 32, K not a power of two), as
// the fused step is: the slot kernel's sum (the full butterfly) and update
// on the copies in LDS, the workers and the broadcast sums written back
// piece after piece.
template <int P, typename T, int R, typename I>
__global__ __launch_bounds__(256) void tensor_sync_staged_kernel(TStepArgs<T> a, int S) {
    constexpr int SPB = 256 / P;  // slot groups per pass
    constexpr int UC = 2 * R;     // passes: S K <= 256 R and K > P / 2 give S < UC SPB
    __shared__ f4 s_x[256 * R], s_g[256 * R];
    const int K = a.K;
    const I s0 = static_cast<I>(tile_of<TC_XCD_RUN_STEP>(blockIdx.x, gridDim.x)) * I(S);
    const I nslot = static_cast<I>(a.nslot);
    const int ns = s0 < nslot ? static_cast<int>(nslot - s0 < I(S) ? nslot - s0 : I(S)) : 0;
    const int np = ns * K;
    const I p0 = s0 * I(K);
    const bool bcast = sizeof(T) == 4 && a.flag;
    f4 vx[R], vg[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int q = threadIdx.x + u * 256;
        if (q < np) {
            vx[u] = load_slot(a.x, p0 + I(q));
            vg[u] = load_slot(static_cast<const T*>(a.g), p0 + I(q));
        }
    }
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int q = threadIdx.x + u * 256;
        if (q < np) {
            s_x[q] = vx[u];
            s_g[q] = vg[u];
        }
    }
    __syncthreads();
    const int i = threadIdx.x % P;
#pragma unroll
    for (int u = 0; u < UC; ++u) {
        if (u * SPB >= ns) break;  // the same for the whole workgroup
        const int jl = u * SPB + static_cast<int>(threadIdx.x) / P;
        const bool live = jl < ns && i < K;
        const int q = jl * K + i;
        const f4 g = live ? s_g[q] : f4(0.0f), x = live ? s_x[q] : f4(0.0f);
        const f4 sum = group_sum4<P>(g);
        if (live) {
            s_x[q] = fma4(f4(-a.s0), sum, x);
            if (bcast) s_g[q] = sum;
        }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < R; ++u) {
        const int q = threadIdx.x + u * 256;
        if (q < np) {
            store_slot(a.x, p0 + I(q), s_x[q]);
            if constexpr (sizeof(T) == 4)
                if (bcast) store_slot(reinterpret_cast<float*>(a.g), p0 + I(q), s_g[q]);
        }
    }
    if (blockIdx.x == gridDim.x - 1) tensor_step_tail<TOp::Sync, P, T>(a);
}

#ifndef TC_TSGD_DENSE
#define TC_TSGD_DENSE 1
#endif
#ifndef TC_TSYNC_STAGED
#define TC_TSYNC_STAGED 1
#endif
template <TOp OP, int P, typename T>
hipError_t run_tstep(const TStepArgs<T>& a, hipStream_t s) {
    if constexpr (OP == TOp::Sync && P >= 32) {
        // bfloat16 gradients: every K between powers of two; binary32: only
        // where more than 7/16 of the slot mapping's lanes would idle
        if (TC_TSYNC_STAGED && a.K != P && (sizeof(T) == 2 || (P - a.K) * 16 > 7 * P)) {
            // slots per workgroup as for the staged fused step (P / 2 < K < P)
            constexpr int R = TC_TEA_STAGED_R;
            const int S = sizeof(T) == 4 ? R * (256 / P) : 256 * R / a.K;
            const int64_t blocks = (a.nslot + S - 1) / S;
            dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
            if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
                hipLaunchKernelGGL((tensor_sync_staged_kernel<P, T, R, uint32_t>), grid, dim3(256), 0, s, a, S);
            else
                hipLaunchKernelGGL((tensor_sync_staged_kernel<P, T, R, int64_t>), grid, dim3(256), 0, s, a, S);
            return hipGetLastError();
        }
    }
    if constexpr (OP == TOp::Sgd) {
        if (TC_TSGD_DENSE && a.K != P) {
            const int64_t blocks = (a.nslot * a.K + 255) / 256;
            dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
            if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
                hipLaunchKernelGGL((tensor_sgd_dense_kernel<T, uint32_t>), grid, dim3(256), 0, s, a);
            else
                hipLaunchKernelGGL((tensor_sgd_dense_kernel<T, int64_t>), grid, dim3(256), 0, s, a);
            return hipGetLastError();
        }
    }
    if constexpr (OP == TOp::Async && sizeof(T) == 4 && P >= 32) {
        if (TC_TASYNC_STAGED && (P >= 64 || (P - a.K) * 4 > P)) {
            constexpr int V = TC_TASYNC_STAGED_V;
            const int KP = a.K | 1;
            const int cap = TC_TASYNC_STAGED_LDS / 16;
            const int S = 64 * V < cap / KP ? 64 * V : cap / KP;
            const int64_t blocks = (a.nslot + S - 1) / S;
            dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
            const size_t lds = static_cast<size_t>(S) * KP * sizeof(f4);
            if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
                hipLaunchKernelGGL((tensor_async_staged_kernel<V, uint32_t>), grid, dim3(256), lds, s, a, S);
            else
                hipLaunchKernelGGL((tensor_async_staged_kernel<V, int64_t>), grid, dim3(256), lds, s, a, S);
            return hipGetLastError();
        }
    }
    if constexpr (OP == TOp::Async && P >= 4 && sizeof(T) == 4) {
        constexpr int U = TC_TASYNC_U;
        constexpr int SPB = 256 / P * U;
        const int64_t blocks = (a.nslot + SPB - 1) / SPB;
        dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
        if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
            hipLaunchKernelGGL((tensor_async_kernel<P, U, uint32_t>), grid, dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((tensor_async_kernel<P, U, int64_t>), grid, dim3(256), 0, s, a);
    } else {
        constexpr int SPB = 256 / P;
        const int64_t blocks = (a.nslot + SPB - 1) / SPB;
        dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
        if ((a.nslot + 1) * a.K * 16 < (int64_t(1) << 32))
            hipLaunchKernelGGL((tensor_step_kernel<OP, P, T, uint32_t>), grid, dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((tensor_step_kernel<OP, P, T, int64_t>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

template <TOp OP, typename T>
hipError_t dispatch_tstep(const TStepArgs<T>& a, hipStream_t s) {
    switch (next_pow2(a.K)) {
#define TC_CASE(p) \
    case p: return run_tstep<OP, p, T>(a, s);
        TC_FOR_P(TC_CASE)
#undef TC_CASE
        default: return hipErrorInvalidValue;
    }
}

template <TOp OP>
hipError_t tstep(int K, float* x, void* g, int g_dtype, float* xc, float s0, int flag, const int32_t* order, int R,
                 int64_t n, hipStream_t s) {
    if (g_dtype == TC_BF16) {
        TStepArgs<uint16_t> a{};
        a.x = x; a.g = static_cast<uint16_t*>(g); a.xc = xc; a.nslot = n / 4; a.n = n; a.s0 = s0; a.K = K; a.flag = flag;
        for (int r = 0; r < R; ++r) a.order[r] = static_cast<uint8_t>(order[r]);
        a.R = R;
        return dispatch_tstep<OP, uint16_t>(a, s);
    }
    TStepArgs<float> a{};
    a.x = x; a.g = static_cast<float*>(g); a.xc = xc; a.nslot = n / 4; a.n = n; a.s0 = s0; a.K = K; a.flag = flag;
    for (int r = 0; r < R; ++r) {
        a.order[r] = static_cast<uint8_t>(order[r]);
        a.exchanged |= uint64_t(1) << order[r];
    }
    a.R = R;
    return dispatch_tstep<OP, float>(a, s);
}

hipError_t launch_tensor_sgd(int K, float* x, const void* g, int g_dtype, float eta, int64_t n, hipStream_t s) {
    return tstep<TOp::Sgd>(K, x, const_cast<void*>(g), g_dtype, nullptr, eta, 0, nullptr, 0, n, s);
}

hipError_t launch_tensor_sync_sgd(int K, float* x, void* g, int g_dtype, float eta, float rescale, int broadcast,
                                  int64_t n, hipStream_t s) {
    const float step = eta * rescale;  // one binary32 rounding, on the host
    return tstep<TOp::Sync>(K, x, g, g_dtype, nullptr, step, g_dtype == TC_BF16 ? 0 : broadcast, nullptr, 0, n, s);
}

hipError_t launch_tensor_elastic_async(int K, float* x, float* xc, const int32_t* order, int R, float alpha, int64_t n,
                                       hipStream_t s) {
    return tstep<TOp::Async>(K, x, nullptr, TC_F32, xc, alpha, 0, order, R, n, s);
}

template <typename T, int U, int PPL>
hipError_t run_tbcast_dense(const void* src, void* dst, int K, int64_t nslot, int64_t n, hipStream_t s) {
    const int64_t blocks = (nslot * K + 256 * U * PPL - 1) / (256 * U * PPL);
    dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
    if ((nslot + 1) * K * 16 < (int64_t(1) << 32))
        hipLaunchKernelGGL((tensor_bcast_dense_kernel<T, U, PPL, uint32_t>), grid, dim3(256), 0, s,
                           static_cast<const T*>(src), static_cast<T*>(dst), nslot, n, K);
    else
        hipLaunchKernelGGL((tensor_bcast_dense_kernel<T, U, PPL, int64_t>), grid, dim3(256), 0, s,
                           static_cast<const T*>(src), static_cast<T*>(dst), nslot, n, K);
    return hipGetLastError();
}

template <int P, typename T>
hipError_t run_tbcast(const void* src, void* dst, int K, int64_t n, hipStream_t s) {
    constexpr int U = TC_TBCAST_UNROLL;
    constexpr int SPB = 256 / P;
    const int64_t nslot = n / 4;
    if (TC_TBCAST_DENSE && K != P) {
        // 8-byte (bf16) pieces go two to a lane from K = 33 on, one to a lane
        // below that: measured on MI355X, two a lane was 10-13% faster at
        // K = 33 and 48 and 3-6% slower at K = 3 to 20
        if constexpr (sizeof(T) == 2)
            if (K > 32) return run_tbcast_dense<T, U, 2>(src, dst, K, nslot, n, s);
        return run_tbcast_dense<T, U, 1>(src, dst, K, nslot, n, s);
    }
    const int64_t blocks = (nslot + SPB * U - 1) / (SPB * U);
    dim3 grid(static_cast<unsigned>(blocks < 1 ? 1 : blocks));
    if ((nslot + 1) * K * 16 < (int64_t(1) << 32))
        hipLaunchKernelGGL((tensor_bcast_kernel<P, T, U, uint32_t>), grid, dim3(256), 0, s, static_cast<const T*>(src),
                           static_cast<T*>(dst), nslot, n, K);
    else
        hipLaunchKernelGGL((tensor_bcast_kernel<P, T, U, int64_t>), grid, dim3(256), 0, s, static_cast<const T*>(src),
                           static_cast<T*>(dst), nslot, n, K);
    return hipGetLastError();
}

hipError_t launch_tensor_broadcast(int K, const void* src, void* dst, int es, int64_t n, hipStream_t s) {
    switch (next_pow2(K)) {
#define TC_CASE(p) \
    case p: return es == 2 ? run_tbcast<p, uint16_t>(src, dst, K, n, s) : run_tbcast<p, uint32_t>(src, dst, K, n, s);
        TC_FOR_P(TC_CASE)
#undef TC_CASE
        default: return hipErrorInvalidValue;
    }
}

}  // namespace tc
