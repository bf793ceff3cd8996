// Device helpers shared by the SFDA kernels (gfx950 / CDNA4, wave64).
//
// Complex matrix products run on the matrix cores in real-block form: for Z = X Y with X
// (rows x K) and Y (K x cols) complex, the real product
//     Z_real[row][2j + q] = sum_{i, p} X_real[row][2i + p] * Ybig[2i + p][2j + q]
// with Ybig[2i][2j] = Re Y, Ybig[2i+1][2j] = -Im Y, Ybig[2i][2j+1] = Im Y,
// Ybig[2i+1][2j+1] = Re Y gives Z with interleaved (re, im) columns -- exactly the complex
// product (the real-coordinate view of complex multiplication, Prop. 3.3), four real
// multiply-adds per complex one and no wasted lanes.
//
// Fragment convention for a 16 x 16 real output tile and a K-block of 16 complex indices
// (32 real K values).  Lane l has tile row/column c = l % 16 and lane group g = l / 16.
//  * The accumulator of a 16x16 MFMA holds D[4 g + r][c] in register r (r = 0..3).
//  * The lane's 8 A values are A8[2 r + p] = part p of X(row = c, i = 4 g + r), and its
//    8 B values are the Ybig entries B8[2 r + p] = Ybig[2 (4 g + r) + p][c].
// Both operands use the same K order, so the sum is independent of how the hardware
// orders K inside an instruction: the bf16 path issues one 16x16x32 MFMA on all 8 values,
// the fp32 path eight 16x16x4 MFMAs, one per value.
//
// A tile held in accumulators whose rows are the K index of a following product converts
// to that product's B fragment in registers: lane (c, g) holds rows 4 g + r of column c and
// its partner lane l ^ 1 holds the other part of the same complex entries.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sfda {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

enum Prec { PREC_F32 = 0, PREC_BF16 = 1 };

// ----------------------------------------------------------------- scalar conversions

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bfloat16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    __device__ __forceinline__ static float load(const float* p, long i) { return p[i]; }
    __device__ __forceinline__ static float2 load2(const float* p, long i) {
        return *reinterpret_cast<const float2*>(p + 2 * i);
    }
    __device__ __forceinline__ static void store2(float* p, long i, float re, float im) {
        *reinterpret_cast<float2*>(p + 2 * i) = make_float2(re, im);
    }
    __device__ __forceinline__ static void store(float* p, long i, float x) { p[i] = x; }
};
template <> struct Elem<uint16_t> {
    __device__ __forceinline__ static float load(const uint16_t* p, long i) {
        return bf16_bits_to_f32(p[i]);
    }
    __device__ __forceinline__ static float2 load2(const uint16_t* p, long i) {
        uint32_t w = *reinterpret_cast<const uint32_t*>(p + 2 * i);
        return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
    }
    __device__ __forceinline__ static void store2(uint16_t* p, long i, float re, float im) {
        uint32_t w = static_cast<uint32_t>(f32_to_bf16_bits(re)) |
                     (static_cast<uint32_t>(f32_to_bf16_bits(im)) << 16);
        *reinterpret_cast<uint32_t*>(p + 2 * i) = w;
    }
    __device__ __forceinline__ static void store(uint16_t* p, long i, float x) {
        p[i] = f32_to_bf16_bits(x);
    }
};

// ----------------------------------------------------------------- branch-free masking

// Keeps a loaded value opaque to the optimiser, so a load that is later masked with a
// select stays unconditional (otherwise it is sunk into a branch and issued -- and waited
// on -- by itself).
__device__ __forceinline__ float pin(float x) { asm volatile("" : "+v"(x)); return x; }
__device__ __forceinline__ float2 pin(float2 x) {
    asm volatile("" : "+v"(x.x), "+v"(x.y));
    return x;
}
__device__ __forceinline__ float masked(bool ok, float x) {
    x = pin(x);
    return ok ? x : 0.f;
}
__device__ __forceinline__ float2 masked(bool ok, float2 x) {
    x = pin(x);
    return ok ? x : make_float2(0.f, 0.f);
}

// ----------------------------------------------------------------- lane exchange

// Value of lane l ^ 1 (DPP quad permutation [1, 0, 3, 2]).
__device__ __forceinline__ float partner(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
}

// ----------------------------------------------------------------- fragments

struct Frag8 { float v[8]; };

// LDS-poison debug build (SFDA_LDS_POISON): fill `bytes` of LDS with all-ones words (NaN as
// float32 and as a bf16 pair), threads tid = 0 .. nthr - 1 together; the caller synchronises
// before and after
__device__ __forceinline__ void lds_poison(void* p, int bytes, int tid, int nthr) {
    uint32_t* w = static_cast<uint32_t*>(p);
    for (int e = tid; e < bytes / 4; e += nthr) w[e] = 0xFFFFFFFFu;
}

// B fragment entries for one complex value y of Y at (i, j), for output column part q:
// q = 0 (real column): (Re y, -Im y); q = 1 (imaginary column): (Im y, Re y).
__device__ __forceinline__ void bpair(Frag8& f, int r, float yr, float yi, int q) {
    f.v[2 * r] = q ? yi : yr;
    f.v[2 * r + 1] = q ? yr : -yi;
}

// B fragment from an accumulator tile whose 16 rows are this product's K-block.
__device__ __forceinline__ Frag8 bfrag_from_acc(const f32x4& acc, int q) {
    Frag8 f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float own = acc[r];
        float oth = partner(own);
        f.v[2 * r] = own;
        f.v[2 * r + 1] = q ? oth : -oth;
    }
    return f;
}

// acc += A * B over one K-block (16 complex = 32 real K values).
template <int P>
__device__ __forceinline__ void mma(f32x4& acc, const Frag8& a, const Frag8& b);

template <>
__device__ __forceinline__ void mma<PREC_F32>(f32x4& acc, const Frag8& a, const Frag8& b) {
#pragma unroll
    for (int s = 0; s < 8; ++s)
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[s], b.v[s], acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mma<PREC_BF16>(f32x4& acc, const Frag8& a, const Frag8& b) {
    bf16x8 x, y;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        x[s] = static_cast<__bf16>(a.v[s]);
        y[s] = static_cast<__bf16>(b.v[s]);
    }
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x, y, acc, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { f32x4 z = {0.f, 0.f, 0.f, 0.f}; return z; }

// ----------------------------------------------------------------- workgroup placement

// Workgroup w of a grid of `heads` x S (head, value-column slice) pairs.  The dispatcher
// hands workgroups to the 8 XCDs round-robin by index and each XCD has its own L2, so the S
// slices of a head -- which read the same q, k, alpha, theta and beta -- are given indices
// 8 S j + 8 s + x (head 8 j + x, slice s): one XCD, one L2.  With a head count that is not a
// multiple of 8 the plain order (head-major) is used.
__device__ __forceinline__ void head_slice(unsigned w, int S, long heads, long& bh, int& sl) {
    if (S > 1 && heads > 0 && (heads & 7) == 0) {
        const unsigned x = w & 7u, q = w >> 3;
        const unsigned j = q / static_cast<unsigned>(S);
        sl = static_cast<int>(q - j * static_cast<unsigned>(S));
        bh = 8L * j + x;
    } else {
        bh = w / S;
        sl = static_cast<int>(w - bh * S);
    }
}

}  // namespace sfda
