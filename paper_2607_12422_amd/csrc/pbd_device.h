// Device-side building blocks for the PEFT-BD kernels on gfx950 (CDNA4).
//
// Data movement is organised around one "fragment": 64 lanes x 16 bytes = 1 KiB,
// the operand one wavefront feeds to a 16x16 MFMA tile.  Lane l owns row (l % 16)
// and lane group g = l / 16 owns EPL consecutive k values (EPL = 16 / sizeof(T):
// 8 bf16 or 4 fp32), so a fragment covers 16 rows x FK = 4 * EPL k values.
// Matrices that are streamed (weights, the K cache) are stored fragment by
// fragment, so one wavefront load instruction reads 1 KiB of contiguous memory.
//
// The MFMA contracts sum over k in an order fixed by the lane layout; operands A
// and B use the same lane -> k assignment, so the contraction is exact up to
// fp32 rounding whatever order the hardware uses internally.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pbd {

typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __bf16 bf16;

constexpr int WAVE = 64;

template <typename T> struct Elt;
template <> struct Elt<float> {
    static constexpr int EPL = 4;      // elements per lane per fragment
    static constexpr int FK = 16;      // k values per fragment
};
template <> struct Elt<bf16> {
    static constexpr int EPL = 8;
    static constexpr int FK = 32;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }  // RNE

// acc += A_frag * B_frag over one fragment's FK k values.
//   a, b: the lane's 16 bytes of the A fragment (row = lane % 16) and of the
//   B fragment (column = lane % 16).
template <typename T> __device__ __forceinline__ void mma_frag(f32x4& acc, const uint4& a, const uint4& b);

template <> __device__ __forceinline__ void mma_frag<bf16>(f32x4& acc, const uint4& a, const uint4& b) {
    bf16x8 av = __builtin_bit_cast(bf16x8, a);
    bf16x8 bv = __builtin_bit_cast(bf16x8, b);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
}

template <> __device__ __forceinline__ void mma_frag<float>(f32x4& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// acc += A * B over 16 k values where each lane supplies 4 consecutive k of its
// row (A) / column (B): lane group g holds k = 4g .. 4g+3.  Used for P.V where
// the B operand (probabilities) comes straight from a 16x16 accumulator.
template <typename T> struct K4;
template <> struct K4<bf16> { typedef uint2 raw; };
template <> struct K4<float> { typedef uint4 raw; };

__device__ __forceinline__ void mma_k4(f32x4& acc, const uint2& a, const f32x4& p) {
    bf16x4 av = __builtin_bit_cast(bf16x4, a);
    bf16x4 bv;
    bv[0] = (bf16)p[0]; bv[1] = (bf16)p[1]; bv[2] = (bf16)p[2]; bv[3] = (bf16)p[3];
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av, bv, acc, 0, 0, 0);
}

__device__ __forceinline__ void mma_k4(f32x4& acc, const uint4& a, const f32x4& p) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), p[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), p[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), p[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), p[3], acc, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Layouts
// ---------------------------------------------------------------------------

// Element offset of (row, k) inside a fragment run: `frag` is the fragment index
// counted in the run, row in [0, 16).
template <typename T>
__device__ __host__ __forceinline__ size_t frag_elem(size_t frag, int row, int k_in_frag) {
    constexpr int EPL = 16 / sizeof(T);
    int g = k_in_frag / EPL, e = k_in_frag % EPL;
    return (frag * 64 + (size_t)(g * 16 + row)) * EPL + e;
}

// Activation operand ("X") of a skinny GEMM: rows m in [0, 16*MT), k in [0, K).
// Fragment (f, mt) sits at index f * MT + mt, so one k step of all m tiles is
// contiguous.
template <typename T>
__device__ __host__ __forceinline__ size_t xfrag_elem(int m, int k, int MT) {
    constexpr int FK = 64 / sizeof(T);
    int f = k / FK;
    return frag_elem<T>((size_t)f * MT + m / 16, m % 16, k % FK);
}

// K cache block: 16 positions x head_dim, fragment ds covers dims [ds*FK, +FK).
template <typename T>
__device__ __host__ __forceinline__ size_t kblock_elem(int key, int dim) {
    constexpr int FK = 64 / sizeof(T);
    return frag_elem<T>(dim / FK, key, dim % FK);
}

// V cache block: 16 positions x head_dim as the A operand of O^T = V^T P^T:
// tile dt covers dims [16 dt, 16 dt + 16); lane (dim % 16) + 16 g holds the
// 4 positions 4g .. 4g+3 of that dim.
__device__ __host__ __forceinline__ size_t vblock_elem(int key, int dim) {
    int dt = dim / 16, g = key / 4, e = key % 4;
    return ((size_t)dt * 64 + (size_t)(g * 16 + dim % 16)) * 4 + e;
}

// Work-group barrier for LDS traffic: waits for this wave's LDS operations
// only, not (as __syncthreads does) for its outstanding global loads, so loads
// issued ahead of time stay in flight across it.  Global data shared through
// memory needs its own wait.
__device__ __forceinline__ void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ---------------------------------------------------------------------------
// Wave reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Reductions over the 16 lanes of a row (DPP: quad swaps, half-row and row mirrors).
__device__ __forceinline__ float row16_sum(float v) {
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));   // lane ^ 1
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));   // lane ^ 2
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));  // half-row mirror
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));  // row mirror
    return v;
}

// Combine lane l with lane l ^ 16 and with lane l ^ 32 (gfx950 permlane swaps).
__device__ __forceinline__ float xrow_max(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float xrow_sum(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// ---------------------------------------------------------------------------
// Per-head QK RMSNorm and RoPE helpers (shared by the attention kernels)
// ---------------------------------------------------------------------------
// Per-head RMSNorm and rotate-half RoPE of one row held by 16 lanes: lane l16
// owns the NP pairs (i, i + HD/2) for i in [NP*l16, NP*l16 + NP), so the
// rotation stays in the lane and the norm is a 16-lane DPP reduction.
template <typename T, int HD>
struct RowPrep {
    static constexpr int HALF = HD / 2;
    static constexpr int NP = HALF / 16;       // pairs per lane (4 or 2)
    typedef float __attribute__((ext_vector_type(NP))) fv;
    typedef float __attribute__((ext_vector_type(2 * NP))) fv2;
    fv lo, hi;
    fv2 cs;                                    // (cos, sin) of the NP pairs
    // vector loads from always-valid addresses; dead rows are zeroed in finish
    __device__ void load(const float* src, const float2* rope_row, int l16) {
        lo = *(const fv*)(src + NP * l16);
        hi = *(const fv*)(src + HALF + NP * l16);
        cs = *(const fv2*)(rope_row + NP * l16);
    }
    // normalise with this lane's gains and rotate; writes the row into dst[HD]
    // as T and returns the lane's values
    __device__ void finish(T* dst, bool live, const float* g_lo, const float* g_hi, bool qk_norm, float eps, int l16,
                           T* out_lo, T* out_hi) {
        values(live, g_lo, g_hi, qk_norm, eps, out_lo, out_hi);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int i = NP * l16 + p;
            dst[i] = out_lo[p];
            dst[i + HALF] = out_hi[p];
        }
    }
    // the lane's normalised and rotated values (dead rows: zeros), no store
    __device__ void values(bool live, const float* g_lo, const float* g_hi, bool qk_norm, float eps, T* out_lo,
                           T* out_hi) {
        float inv = live ? 1.f : 0.f;
        if (qk_norm) {
            float ss = 0.f;
#pragma unroll
            for (int p = 0; p < NP; ++p) ss += lo[p] * lo[p] + hi[p] * hi[p];
            inv = live ? rsqrtf(row16_sum(ss) / (float)HD + eps) : 0.f;
        }
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const float y0 = lo[p] * inv * g_lo[p], y1 = hi[p] * inv * g_hi[p];
            const float c = cs[2 * p], sn = cs[2 * p + 1];
            out_lo[p] = from_f32<T>(y0 * c - y1 * sn);
            out_hi[p] = from_f32<T>(y1 * c + y0 * sn);
        }
    }
};

// this lane's RMSNorm gains: raw loads now, conversion at first use
template <typename T, int HD>
struct Gains {
    static constexpr int NP = RowPrep<T, HD>::NP, HALF = HD / 2;
    typedef T __attribute__((ext_vector_type(NP))) tv;
    tv rlo, rhi;
    __device__ void load(const void* gain, int l16) {
        rlo = *(const tv*)((const T*)gain + NP * l16);
        rhi = *(const tv*)((const T*)gain + HALF + NP * l16);
    }
    __device__ void get(bool qk_norm, float* g_lo, float* g_hi) const {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            g_lo[p] = qk_norm ? to_f32(rlo[p]) : 1.f;
            g_hi[p] = qk_norm ? to_f32(rhi[p]) : 1.f;
        }
    }
};

}  // namespace pbd
