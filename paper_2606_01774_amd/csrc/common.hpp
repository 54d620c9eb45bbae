// common.hpp -- device helpers shared by the HIP kernels of the block-diffusion Gated
// Delta Rule on gfx950 (CDNA4): element types, MFMA tile products over LDS,
// conversions, barriers.
//
// MFMA operand convention: a 16x16 output tile C += A * B where A is 16 x K and B is
// given transposed (16 x K); both live in LDS with K contiguous.  Lane l holds
// C[4*(l>>4) + i][l & 15] in accumulator element i.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdgdn {

typedef float f32x4 __attribute__((ext_vector_type(4)));
// 16-byte chunk of raw data; a native vector (not HIP's uint4 class) so that selects
// stay in registers.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

template <typename E> struct Mma;

// bf16 operands, fp32 accumulate: v_mfma_f32_16x16x32_bf16 (8 operands per lane).
// Products of bf16 inputs are exact in the fp32 accumulator.
template <> struct Mma<__bf16> {
    static constexpr int kStep = 32;
    static constexpr int kPerLane = 8;
    static constexpr int kPad = 8;  // LDS row padding in elements (16 bytes)
    typedef bf16x8 frag;
    static __device__ __forceinline__ frag load(const __bf16 *p)
    {
        return *reinterpret_cast<const bf16x8 *>(p);
    }
    static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

// fp16 operands, fp32 accumulate: v_mfma_f32_16x16x32_f16 (8 operands per lane).  The
// bf16 inputs are staged as fp16 (exact for |x| in [2^-14, 2^15]); every rounded
// intermediate operand (state, T, masked Q K^T, Delta) then carries 11 significant
// bits instead of bf16's 8, at the same MFMA rate.
template <> struct Mma<_Float16> {
    static constexpr int kStep = 32;
    static constexpr int kPerLane = 8;
    static constexpr int kPad = 8;  // LDS row padding in elements (16 bytes)
    typedef f16x8 frag;
    static __device__ __forceinline__ frag load(const _Float16 *p)
    {
        return *reinterpret_cast<const f16x8 *>(p);
    }
    static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

// fp32 operands: v_mfma_f32_16x16x4_f32 (one operand per lane).
template <> struct Mma<float> {
    static constexpr int kStep = 4;
    static constexpr int kPerLane = 1;
    static constexpr int kPad = 4;
    typedef float frag;
    static __device__ __forceinline__ frag load(const float *p) { return *p; }
    static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
};

template <typename E> __device__ __forceinline__ E to_e(float x);
template <> __device__ __forceinline__ __bf16 to_e<__bf16>(float x) { return (__bf16)x; }
template <> __device__ __forceinline__ _Float16 to_e<_Float16>(float x) { return (_Float16)x; }
template <> __device__ __forceinline__ float to_e<float>(float x) { return x; }
__device__ __forceinline__ float to_f(__bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f(_Float16 x) { return (float)x; }
__device__ __forceinline__ float to_f(float x) { return x; }

// A 16-byte chunk of input elements re-encoded as operand elements of the same size.
template <typename In, typename Op> __device__ __forceinline__ u32x4 to_operand(u32x4 raw)
{
    static_assert(sizeof(In) == sizeof(Op), "same element size");
    if constexpr (__is_same(In, Op)) {
        return raw;
    } else {
        constexpr int N = 16 / sizeof(In);
        In src[N];
        Op dst[N];
        __builtin_memcpy(src, &raw, 16);
#pragma unroll
        for (int e = 0; e < N; ++e) dst[e] = to_e<Op>(to_f(src[e]));
        u32x4 out;
        __builtin_memcpy(&out, dst, 16);
        return out;
    }
}

// Four consecutive elements to LDS (8-byte store for 16-bit types, 16-byte for fp32).
__device__ __forceinline__ void st4(_Float16 *p, float a, float b, float c, float d)
{
    f16x4 v = {(_Float16)a, (_Float16)b, (_Float16)c, (_Float16)d};
    *reinterpret_cast<f16x4 *>(p) = v;
}
__device__ __forceinline__ void st4(__bf16 *p, float a, float b, float c, float d)
{
    bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4 *>(p) = v;
}
__device__ __forceinline__ void st4(float *p, float a, float b, float c, float d)
{
    f32x4 v = {a, b, c, d};
    *reinterpret_cast<f32x4 *>(p) = v;
}

// One 16x16x16 step with 4 operands per lane (K = 16 tails of 16-bit products).
__device__ __forceinline__ f32x4 mma16(const _Float16 *a, const _Float16 *b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16f16(*reinterpret_cast<const f16x4 *>(a),
                                                  *reinterpret_cast<const f16x4 *>(b), c, 0, 0, 0);
}
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4 mma16(const __bf16 *a, const __bf16 *b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(*reinterpret_cast<const s16x4 *>(a),
                                                     *reinterpret_cast<const s16x4 *>(b), c, 0, 0, 0);
}

// C(16x16) += A(16 x K) * Bt(16 x K)^T, operands in LDS with K contiguous.  For 16-bit
// operands a K that is not a multiple of 32 ends with one 16x16x16 step (4 operands
// per lane) so no operand is read past K.
template <typename E, int K>
__device__ __forceinline__ f32x4 tile_mma(f32x4 acc, const E *A, int lda, const E *Bt, int ldb,
                                          int lane)
{
    constexpr int KS = Mma<E>::kStep;
    constexpr int KMAIN = K - K % KS;
    const int r = lane & 15, ko = (lane >> 4) * Mma<E>::kPerLane;
    const E *a = A + r * lda + ko;
    const E *b = Bt + r * ldb + ko;
#pragma unroll
    for (int k0 = 0; k0 < KMAIN; k0 += KS)
        acc = Mma<E>::mma(Mma<E>::load(a + k0), Mma<E>::load(b + k0), acc);
    if constexpr (KMAIN != K) {
        static_assert(sizeof(E) == 2 && K - KMAIN == 16, "16-bit tail of 16");
        const int k4 = (lane >> 4) * 4;
        acc = mma16(A + r * lda + KMAIN + k4, Bt + r * ldb + KMAIN + k4, acc);
    }
    return acc;
}

// C(16x16) += A(16 x K) * Bt(16 x K)^T where A is the transpose of a row-major LDS
// matrix R (A[m][k] = R[k][m], row stride ldr): the operand is gathered element by
// element, so R needs no transposed copy.
template <typename E, int K>
__device__ __forceinline__ f32x4 tile_mma_at(f32x4 acc, const E *R, int ldr, const E *Bt, int ldb,
                                             int lane)
{
    constexpr int KS = Mma<E>::kStep, KP = Mma<E>::kPerLane;
    constexpr int KMAIN = K - K % KS;
    const int r = lane & 15, ko = (lane >> 4) * KP;
    const E *a = R + ko * ldr + r;
    const E *b = Bt + r * ldb + ko;
#pragma unroll
    for (int k0 = 0; k0 < KMAIN; k0 += KS) {
        typename Mma<E>::frag fa;
        if constexpr (KP == 1) {
            fa = a[k0 * ldr];
        } else {
#pragma unroll
            for (int j = 0; j < KP; ++j) fa[j] = a[(k0 + j) * ldr];
        }
        acc = Mma<E>::mma(fa, Mma<E>::load(b + k0), acc);
    }
    if constexpr (KMAIN != K) {
        static_assert(sizeof(E) == 2 && K - KMAIN == 16, "16-bit tail of 16");
        const int k4 = (lane >> 4) * 4;
        E a4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) a4[j] = R[(KMAIN + k4 + j) * ldr + r];
        acc = mma16(a4, Bt + r * ldb + KMAIN + k4, acc);
    }
    return acc;
}

// C(16x16) += A (B1 + B2)^T with each A fragment loaded once: the B operand given as
// a hi + lo pair (an fp32 value carried in two 16-bit operands).
template <typename E, int K>
__device__ __forceinline__ f32x4 tile_mma2(f32x4 acc, const E *A, int lda, const E *B1, const E *B2,
                                           int ldb, int lane)
{
    constexpr int KS = Mma<E>::kStep;
    constexpr int KMAIN = K - K % KS;
    const int r = lane & 15, ko = (lane >> 4) * Mma<E>::kPerLane;
    const E *a = A + r * lda + ko;
    const E *b1 = B1 + r * ldb + ko;
    const E *b2 = B2 + r * ldb + ko;
#pragma unroll
    for (int k0 = 0; k0 < KMAIN; k0 += KS) {
        const typename Mma<E>::frag fa = Mma<E>::load(a + k0);
        acc = Mma<E>::mma(fa, Mma<E>::load(b2 + k0), acc);
        acc = Mma<E>::mma(fa, Mma<E>::load(b1 + k0), acc);
    }
    if constexpr (KMAIN != K) {
        static_assert(sizeof(E) == 2 && K - KMAIN == 16, "16-bit tail of 16");
        const int k4 = (lane >> 4) * 4;
        acc = mma16(A + r * lda + KMAIN + k4, B2 + r * ldb + KMAIN + k4, acc);
        acc = mma16(A + r * lda + KMAIN + k4, B1 + r * ldb + KMAIN + k4, acc);
    }
    return acc;
}

// tile_mma_at with the B operand given as a hi + lo pair.
template <typename E, int K>
__device__ __forceinline__ f32x4 tile_mma_at2(f32x4 acc, const E *R, int ldr, const E *B1, const E *B2,
                                              int ldb, int lane)
{
    constexpr int KS = Mma<E>::kStep, KP = Mma<E>::kPerLane;
    constexpr int KMAIN = K - K % KS;
    const int r = lane & 15, ko = (lane >> 4) * KP;
    const E *a = R + ko * ldr + r;
    const E *b1 = B1 + r * ldb + ko;
    const E *b2 = B2 + r * ldb + ko;
#pragma unroll
    for (int k0 = 0; k0 < KMAIN; k0 += KS) {
        typename Mma<E>::frag fa;
#pragma unroll
        for (int j = 0; j < KP; ++j) fa[j] = a[(k0 + j) * ldr];
        acc = Mma<E>::mma(fa, Mma<E>::load(b2 + k0), acc);
        acc = Mma<E>::mma(fa, Mma<E>::load(b1 + k0), acc);
    }
    if constexpr (KMAIN != K) {
        static_assert(sizeof(E) == 2 && K - KMAIN == 16, "16-bit tail of 16");
        const int k4 = (lane >> 4) * 4;
        E a4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) a4[j] = R[(KMAIN + k4 + j) * ldr + r];
        acc = mma16(a4, B2 + r * ldb + KMAIN + k4, acc);
        acc = mma16(a4, B1 + r * ldb + KMAIN + k4, acc);
    }
    return acc;
}

// ------------------------------------------------------------------ quad operands
// Lane (g = lane >> 4, r = lane & 15) of a 16x16 MFMA tile can hold, for operand row r
// (a row of A, a column of B), the four values at k = 4g .. 4g+3 of a 16-wide k-block:
// a "quad".  An accumulator tile is held the same way (lane (g, n) has C[4g + i][n]), so
// an accumulator feeds the next product straight from registers: as a B operand whose
// k runs over its rows, or as the A operand of its transpose.  A product over
// K = 16 NKB takes NKB quads per operand and lane; since any fixed assignment of the
// k values to MFMA operand slots yields the same sum, two k-blocks fill one 16x16x32
// step (16-bit types) and a k-block is four 16x16x4 steps (fp32).
template <typename E> struct QuadOf;
template <> struct QuadOf<_Float16> { typedef f16x4 type; };
template <> struct QuadOf<float> { typedef f32x4 type; };
template <typename E> using Quad = typename QuadOf<E>::type;

template <typename E> __device__ __forceinline__ Quad<E> ld_quad(const E *p)
{
    return *reinterpret_cast<const Quad<E> *>(p);
}
template <typename E> __device__ __forceinline__ void st_quad(E *p, Quad<E> q)
{
    *reinterpret_cast<Quad<E> *>(p) = q;
}
template <typename E> __device__ __forceinline__ Quad<E> quad_of(f32x4 a);
template <> __device__ __forceinline__ f16x4 quad_of<_Float16>(f32x4 a)
{
    return f16x4{(_Float16)a[0], (_Float16)a[1], (_Float16)a[2], (_Float16)a[3]};
}
template <> __device__ __forceinline__ f32x4 quad_of<float>(f32x4 a) { return a; }

// Quads of row (lane & 15) of the row-major LDS matrix M (row stride ld), k-blocks
// 0 .. NKB-1 starting at M's first column.  Each quad is its own 8-byte LDS read: with
// rows 16 bytes past a multiple of 256 bytes these are free of bank conflicts, while the
// paired two-address reads the compiler would otherwise form from them are not (8
// conflict cycles per pair on gfx950); the volatile access keeps them unpaired.
template <typename E, int NKB>
__device__ __forceinline__ void ld_quads(Quad<E> (&q)[NKB], const E *M, int ld, int lane)
{
    typedef const __attribute__((address_space(3))) volatile Quad<E> *LQ;
    const E *p = M + (lane & 15) * ld + 4 * (lane >> 4);
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) q[kb] = *(LQ)(p + 16 * kb);
}

// acc += sum over k-blocks kb of A_kb B_kb.
template <typename E, int NKB>
__device__ __forceinline__ f32x4 mma_q(f32x4 acc, const Quad<E> (&a)[NKB], const Quad<E> (&b)[NKB])
{
    if constexpr (sizeof(E) == 2) {
#pragma unroll
        for (int u = 0; u + 1 < NKB; u += 2) {
            const f16x8 a8 = __builtin_shufflevector(a[u], a[u + 1], 0, 1, 2, 3, 4, 5, 6, 7);
            const f16x8 b8 = __builtin_shufflevector(b[u], b[u + 1], 0, 1, 2, 3, 4, 5, 6, 7);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a8, b8, acc, 0, 0, 0);
        }
        if constexpr (NKB % 2) acc = __builtin_amdgcn_mfma_f32_16x16x16f16(a[NKB - 1], b[NKB - 1], acc, 0, 0, 0);
    } else {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[kb][i], b[kb][i], acc, 0, 0, 0);
    }
    return acc;
}

// C(16x16) += A(16 x K) * B(K x 16), fp32, both row-major in LDS (used by the solve).
__device__ __forceinline__ f32x4 tile_mma_rr(f32x4 acc, const float *A, int lda, const float *B,
                                             int ldb, int K, int lane)
{
    const int m = lane & 15, kk = lane >> 4;
    for (int k0 = 0; k0 < K; k0 += 4)
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A[m * lda + k0 + kk], B[(k0 + kk) * ldb + m],
                                                   acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations, then
// s_barrier.  Unlike __syncthreads it does not wait for outstanding global loads or
// stores (no global memory is exchanged between threads inside a block step), so a
// prefetch issued before it stays in flight.  The "memory" clobber keeps the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until all of this wave's global loads have returned (s_waitcnt vmcnt(0) on
// gfx9-family encodings: vmcnt = 0, expcnt and lgkmcnt left at their maxima).  Used
// once after loads issued before a loop, so the loop's own waits only ever count the
// loop's loads.
__device__ __forceinline__ void wait_global_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// 2^x with the hardware v_exp_f32 (arguments here are block-local gate differences,
// within [-12, 0]).
__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Lower-triangular tile index -> (bi, bj), bi >= bj, row-major over bi.
__device__ __forceinline__ void tri_decode(int l, int &bi, int &bj)
{
    bi = 0;
    while (l > bi) {
        l -= bi + 1;
        ++bi;
    }
    bj = l;
}

}  // namespace bdgdn
