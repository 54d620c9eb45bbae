// engine.hpp -- device building blocks of the block-diffusion Gated Delta Rule on
// gfx950 (CDNA4): MFMA tile products over LDS, the block-local UT transform, and the
// per-block two-stream step shared by the training and serving kernels.
//
// Mathematics (FLARE, arXiv 2606.01774; Appendix eq. per-step-fwd, eq. chunk-state,
// eq. f-blk, eq. noisy-block-fwd).  For one block of n positions that starts from the
// clean state S0 (d_k x d_v) and local cumulative log-gates G_r (G_0 = 0):
//   gamma_r = exp(G_r),  A_ri = beta_r (gamma_r / gamma_i) (k_r . k_i)  (i < r)
//   T = (I + A)^{-1} diag(beta)                        (the UT / WY transform)
//   Delta = T (V - diag(gamma) K S0)                    (rows = the paper's delta_t)
//   O     = s [ diag(gamma) Q S0 + (Q K^T o Mc) Delta ],  Mc_ri = gamma_r/gamma_i, i <= r
//   S_n   = gamma_n S0 + K^T diag(gamma_n / gamma) Delta
// and for the noisy block seeded with the same S0 (block-end readout):
//   Delta~ = T~ (V~ - diag(gamma~) K~ S0)
//   O~     = s [ gamma~_n Q~ S0 + (Q~ K~^T diag(gamma~_n / gamma~)) Delta~ ].
// These are exact rewritings of the sequential recurrence (induction on
// S_r = gamma_r S0 + sum_{i<=r} (gamma_r/gamma_i) k_i delta_i^T); only
// exponentials of block-local differences are ever formed.
//
// MFMA operand convention: a 16x16 output tile C += A * B where A is 16 x K and B is
// given transposed (16 x K); both live in LDS with K contiguous.  Lane l holds
// C[4*(l>>4) + i][l & 15] in accumulator element i.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdgdn {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLog2e = 1.4426950408889634f;

template <typename E> struct Mma;

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
template <typename In, typename Op> __device__ __forceinline__ uint4 to_operand(uint4 raw)
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
        uint4 out;
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
__device__ __forceinline__ void st4(float *p, float a, float b, float c, float d)
{
    f32x4 v = {a, b, c, d};
    *reinterpret_cast<f32x4 *>(p) = v;
}

// C(16x16) += A(16 x K) * Bt(16 x K)^T, operands in LDS with K contiguous.  For fp16
// a K that is not a multiple of 32 ends with one v_mfma_f32_16x16x16_f16 step
// (4 operands per lane) so no operand is read past K.
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
        static_assert(sizeof(E) == 2 && K - KMAIN == 16, "fp16 tail of 16");
        const int k4 = (lane >> 4) * 4;
        const f16x4 a4 = *reinterpret_cast<const f16x4 *>(A + r * lda + KMAIN + k4);
        const f16x4 b4 = *reinterpret_cast<const f16x4 *>(Bt + r * ldb + KMAIN + k4);
        acc = __builtin_amdgcn_mfma_f32_16x16x16f16(a4, b4, acc, 0, 0, 0);
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

// ---------------------------------------------------------------------------------
// Shared-memory layout of one workgroup.  Buffers whose lifetimes do not overlap
// within a block share the region U:
//   phase load..gram : the q/k row buffers
//   phase epilogue..T: A (fp32, becomes (I+A)^{-1} in place), the solve's scratch,
//                      T, and D = V - diag(gamma) K S0 (transposed)
//   phase delta..end : Delta (transposed), decayed Delta, noisy Delta~
// ---------------------------------------------------------------------------------
template <typename E, int DK, int BV, int LP, bool CL, bool CO, bool NZ>
struct Layout {
    static_assert(LP % 16 == 0 && LP >= 16 && LP <= 64, "block tile");
    static_assert(DK % 32 == 0 && BV % 16 == 0, "tile sizes");
    static constexpr int SZ = (int)sizeof(E);
    static constexpr int PE = Mma<E>::kPad;
    static constexpr int RS = DK + PE;   // stride of [token][d_k] rows and of ST [v][d_k]
    static constexpr int TS = LP + PE;   // stride of [*][token] buffers
    static constexpr int VS = BV + PE;   // stride of the staged V tile [token][v]
    static constexpr int FS = LP + 4;    // fp32 stride of A / (I+A)^{-1}
    static constexpr int NB = LP / 16;
    static constexpr int NVB = BV / 16;
    static constexpr int NSOLVE = (CL ? 1 : 0) + (NZ ? 1 : 0);
    static constexpr int NROWS = (CL ? 1 : 0) + (CO ? 1 : 0) + (NZ ? 2 : 0);
    // row-buffer slots
    static constexpr int SLOT_K = 0;
    static constexpr int SLOT_Q = 1;
    static constexpr int SLOT_KN = CL ? (CO ? 2 : 1) : 0;
    static constexpr int SLOT_QN = SLOT_KN + 1;

    static constexpr int al(int x) { return (x + 15) & ~15; }
    static constexpr int mx(int a, int b) { return a > b ? a : b; }

    static constexpr int ROWS_B = al(LP * RS * SZ);                 // one row set
    static constexpr int A_B = al(LP * FS * 4);                     // one A matrix
    static constexpr int Y_B = NSOLVE * (NB > 1 ? NB - 1 : 1) * 256 * 4;
    static constexpr int TM_B = al(LP * TS * SZ);                   // one T/P/R matrix
    static constexpr int DT_B = al(BV * TS * SZ);                   // one [v][token] tile
    static constexpr int NPOST = (CL ? 2 : 0) + (NZ ? 1 : 0);        // Delta, decayed Delta, Delta~
    static constexpr int OFF_A = 0;
    static constexpr int OFF_Y = NSOLVE * A_B;
    static constexpr int OFF_POST = 0;                               // over A after the solve
    static constexpr int OFF_T = al(mx(OFF_Y + Y_B, NPOST * DT_B));
    static constexpr int OFF_D = OFF_T + NSOLVE * TM_B;
    static constexpr int U_B = al(mx(NROWS * ROWS_B, OFF_D + NSOLVE * DT_B));

    static constexpr int OFF_U = 0;
    static constexpr int OFF_KT = OFF_U + U_B;
    static constexpr int KT_B = CL ? al(DK * TS * SZ) : 0;
    static constexpr int OFF_ST = OFF_KT + KT_B;
    static constexpr int ST_B = al(BV * RS * SZ);
    static constexpr int OFF_V = OFF_ST + ST_B;
    static constexpr int V_B = al(LP * VS * SZ);
    static constexpr int OFF_PR = OFF_V + NSOLVE * V_B;
    static constexpr int NPR = (CO ? 1 : 0) + (NZ ? 1 : 0);
    static constexpr int OFF_GATES = OFF_PR + NPR * TM_B;
    static constexpr int BYTES = OFF_GATES + 4 * 64 * 4;
};

// Gate slots in the gate area: 0 = g (becomes G*log2e), 1 = beta, 2 = gn (-> Gn*log2e), 3 = betan.
constexpr int GS_G = 0, GS_B = 1, GS_GN = 2, GS_BN = 3;

// Pointers of one block's rows in global memory (row r of a tensor is base + r*stride).
template <typename In, typename Out> struct BlockIO {
    const In *k, *q, *v, *kn, *qn, *vn;  // first row of the block (q/k: head hq; v: head h, col v0)
    const float *g, *beta, *gn, *betan;  // first row of the block (head h)
    Out *o, *on;                         // first row (head h, col v0)
    long qk_stride, v_stride, gate_stride;  // elements between consecutive rows
    int nvalid;                          // rows of this block that exist (<= L)
};

// In: element type of q, k, v in global memory; E: MFMA operand type in LDS (same size
// as In); Out: element type of the outputs.
template <typename In, typename E, typename Out, int DK, int BV, int LP, bool CL, bool CO, bool NZ>
struct Engine {
    static_assert(sizeof(In) == sizeof(E), "inputs are staged chunk for chunk");
    typedef Layout<E, DK, BV, LP, CL, CO, NZ> Ly;
    typedef BlockIO<In, Out> IO;
    static constexpr int NB = Ly::NB, NVB = Ly::NVB;
    static constexpr int NL = NB * (NB + 1) / 2;  // lower tiles incl. diagonal
    static constexpr int NF = NB * NB;
    static constexpr int NX = NB * NVB;           // tiles of an LP x BV product
    static constexpr int NS = (DK / 16) * NVB;    // tiles of the d_k x BV state
    // phase-G list: [KK lower][QK full][KnKn lower][QnKn full][X1][X3]
    static constexpr int G_KK = CL ? NL : 0;
    static constexpr int G_QK = CO ? NF : 0;
    static constexpr int G_KN = NZ ? NL : 0;
    static constexpr int G_QN = NZ ? NF : 0;
    static constexpr int G_X1 = CL ? NX : 0;
    static constexpr int G_X3 = NZ ? NX : 0;
    static constexpr int NG = G_KK + G_QK + G_KN + G_QN + G_X1 + G_X3;
    static constexpr int NGW = (NG + kWaves - 1) / kWaves;
    static constexpr int NXW = (NX + kWaves - 1) / kWaves;
    static constexpr int NSW = (NS + kWaves - 1) / kWaves;
    static constexpr int ND = (CL ? NX : 0) + (NZ ? NX : 0);
    static constexpr int NDW = (ND + kWaves - 1) / kWaves;
    static constexpr int EPC = 16 / Ly::SZ;       // elements per 16-byte chunk
    static constexpr int CPR = DK / EPC;
    static constexpr int RCH = LP * CPR;
    static constexpr int RPT = (RCH + kThreads - 1) / kThreads;
    static constexpr int VCPR = BV / EPC;
    static constexpr int VCH = LP * VCPR;
    static constexpr int VPT = (VCH + kThreads - 1) / kThreads;

    unsigned char *smem;
    int tid, lane, wave;

    __device__ E *rows(int slot) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + slot * Ly::ROWS_B); }
    __device__ float *amat(int m) const { return reinterpret_cast<float *>(smem + Ly::OFF_U + Ly::OFF_A + m * Ly::A_B); }
    __device__ float *ytmp(int p) const { return reinterpret_cast<float *>(smem + Ly::OFF_U + Ly::OFF_Y) + p * 256; }
    __device__ E *tmat(int m) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + Ly::OFF_T + m * Ly::TM_B); }
    __device__ E *dmat(int m) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + Ly::OFF_D + m * Ly::DT_B); }
    // post-solve [v][token] buffers: 0 = Delta, 1 = decayed Delta (clean), 2 or 0 = Delta~
    __device__ E *post(int i) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + Ly::OFF_POST + i * Ly::DT_B); }
    __device__ E *kt() const { return reinterpret_cast<E *>(smem + Ly::OFF_KT); }
    __device__ E *st() const { return reinterpret_cast<E *>(smem + Ly::OFF_ST); }
    __device__ E *vs(int m) const { return reinterpret_cast<E *>(smem + Ly::OFF_V + m * Ly::V_B); }
    __device__ E *pm() const { return reinterpret_cast<E *>(smem + Ly::OFF_PR); }
    __device__ E *rm() const { return reinterpret_cast<E *>(smem + Ly::OFF_PR + (CO ? Ly::TM_B : 0)); }
    __device__ float *gates(int s) const { return reinterpret_cast<float *>(smem + Ly::OFF_GATES) + s * 64; }

    static constexpr int SOLVE_N = Ly::NSOLVE;   // solve matrix index: 0 = clean (if CL), last = noisy
    static constexpr int MAT_C = 0;
    static constexpr int MAT_N = CL ? 1 : 0;
    static constexpr int POST_N = CL ? 2 : 0;

    __device__ Engine(unsigned char *s) : smem(s)
    {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = wave_id();
    }

    // ----------------------------------------------------------------- state I/O
    // Load fp32 state tile [d_k][v0..v0+BV) of row stride dv into accumulator layout
    // (tile t = (bk, bc) holds S[16bk + 4(l>>4) + i][16bc + (l&15)]).  src == NULL -> 0.
    __device__ void load_state(f32x4 (&S)[NSW], const float *src, int dv) const
    {
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * kWaves;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            if (t < NS && src) {
                const int bk = t / NVB, bc = t % NVB;
                const float *p = src + (long)(16 * bk + 4 * (lane >> 4)) * dv + 16 * bc + (lane & 15);
                acc[0] = p[0];
                acc[1] = p[dv];
                acc[2] = p[2 * dv];
                acc[3] = p[3 * dv];
            }
            S[s] = acc;
        }
    }
    __device__ void store_state(const f32x4 (&S)[NSW], float *dst, int dv) const
    {
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * kWaves;
            if (t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                float *p = dst + (long)(16 * bk + 4 * (lane >> 4)) * dv + 16 * bc + (lane & 15);
                p[0] = S[s][0];
                p[dv] = S[s][1];
                p[2 * dv] = S[s][2];
                p[3 * dv] = S[s][3];
            }
        }
    }
    // S^T (MFMA operand, dtype E) into LDS: ST[v][d_k].
    __device__ void write_st(const f32x4 (&S)[NSW]) const
    {
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * kWaves;
            if (t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                E *p = st() + (16 * bc + (lane & 15)) * Ly::RS + 16 * bk + 4 * (lane >> 4);
                st4(p, S[s][0], S[s][1], S[s][2], S[s][3]);
            }
        }
    }

    // ----------------------------------------------------------------- phase L
    // Global -> LDS for one block: q/k rows (and K transposed), the V tiles, gates.
    // Rows at or past nvalid are zero: identity positions (k = 0, g = 0, beta = 0).
    __device__ void load_block(const IO &io) const
    {
        constexpr int NR = Ly::NROWS;
        const In *src[4] = {nullptr, nullptr, nullptr, nullptr};
        if (CL) src[Ly::SLOT_K] = io.k;
        if (CO) src[Ly::SLOT_Q] = io.q;
        if (NZ) {
            src[Ly::SLOT_KN] = io.kn;
            src[Ly::SLOT_QN] = io.qn;
        }
        uint4 rb[NR][RPT];
        const uint4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int rs = 0; rs < NR; ++rs)
#pragma unroll
            for (int s = 0; s < RPT; ++s) {
                const int c = tid + s * kThreads;
                const int t = c / CPR, cc = c % CPR;
                rb[rs][s] = (c < RCH && t < io.nvalid)
                                ? to_operand<In, E>(*reinterpret_cast<const uint4 *>(src[rs] + t * io.qk_stride + cc * EPC))
                                : zero;
            }
        const In *vsrc[2] = {CL ? io.v : io.vn, io.vn};
        uint4 vb[Ly::NSOLVE][VPT];
#pragma unroll
        for (int m = 0; m < Ly::NSOLVE; ++m)
#pragma unroll
            for (int s = 0; s < VPT; ++s) {
                const int c = tid + s * kThreads;
                const int t = c / VCPR, cc = c % VCPR;
                vb[m][s] = (c < VCH && t < io.nvalid)
                               ? to_operand<In, E>(*reinterpret_cast<const uint4 *>(vsrc[m] + t * io.v_stride + cc * EPC))
                               : zero;
            }
        float gv = 0.f;
        {
            const int which = tid / LP, t = tid % LP;
            const float *gp = nullptr;
            if (which == GS_G && CL) gp = io.g;
            if (which == GS_B && CL) gp = io.beta;
            if (which == GS_GN && NZ) gp = io.gn;
            if (which == GS_BN && NZ) gp = io.betan;
            if (which < 4 && gp && t < io.nvalid) gv = gp[t * io.gate_stride];
        }
        // LDS writes
#pragma unroll
        for (int rs = 0; rs < NR; ++rs)
#pragma unroll
            for (int s = 0; s < RPT; ++s) {
                const int c = tid + s * kThreads;
                if (c < RCH) {
                    const int t = c / CPR, cc = c % CPR;
                    *reinterpret_cast<uint4 *>(rows(rs) + t * Ly::RS + cc * EPC) = rb[rs][s];
                }
            }
        if (CL) {
#pragma unroll
            for (int s = 0; s < RPT; ++s) {
                const int c = tid + s * kThreads;
                if (c < RCH) {
                    const int t = c / CPR, cc = c % CPR;
                    E tmp[EPC];
                    __builtin_memcpy(tmp, &rb[Ly::SLOT_K][s], 16);
#pragma unroll
                    for (int e = 0; e < EPC; ++e) kt()[(cc * EPC + e) * Ly::TS + t] = tmp[e];
                }
            }
        }
#pragma unroll
        for (int m = 0; m < Ly::NSOLVE; ++m)
#pragma unroll
            for (int s = 0; s < VPT; ++s) {
                const int c = tid + s * kThreads;
                if (c < VCH) {
                    const int t = c / VCPR, cc = c % VCPR;
                    *reinterpret_cast<uint4 *>(vs(m) + t * Ly::VS + cc * EPC) = vb[m][s];
                }
            }
        if (tid < 4 * LP) gates(tid / LP)[tid % LP] = gv;
    }

    // In-place inclusive scan of a gate slot (times log2 e), by one wave.
    __device__ void scan_gates(int slot) const
    {
        float *gp = gates(slot);
        float x = lane < LP ? gp[lane] * kLog2e : 0.f;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const float y = __shfl_up(x, d, 64);
            if (lane >= d) x += y;
        }
        if (lane < LP) gp[lane] = x;
    }

    // ----------------------------------------------------------------- phase G
    // Which operands a phase-G list entry multiplies; K = DK for all of them.
    __device__ void g_decode(int idx, int &kind, int &bi, int &bj, const E *&A, const E *&B) const
    {
        int l = idx;
        kind = 0;
        if (l < G_KK) { tri_decode(l, bi, bj); kind = 0; A = rows(Ly::SLOT_K) + 16 * bi * Ly::RS; B = rows(Ly::SLOT_K) + 16 * bj * Ly::RS; return; }
        l -= G_KK;
        if (l < G_QK) { bi = l / NB; bj = l % NB; kind = 1; A = rows(Ly::SLOT_Q) + 16 * bi * Ly::RS; B = rows(Ly::SLOT_K) + 16 * bj * Ly::RS; return; }
        l -= G_QK;
        if (l < G_KN) { tri_decode(l, bi, bj); kind = 2; A = rows(Ly::SLOT_KN) + 16 * bi * Ly::RS; B = rows(Ly::SLOT_KN) + 16 * bj * Ly::RS; return; }
        l -= G_KN;
        if (l < G_QN) { bi = l / NB; bj = l % NB; kind = 3; A = rows(Ly::SLOT_QN) + 16 * bi * Ly::RS; B = rows(Ly::SLOT_KN) + 16 * bj * Ly::RS; return; }
        l -= G_QN;
        if (l < G_X1) { bi = l / NVB; bj = l % NVB; kind = 4; A = rows(Ly::SLOT_K) + 16 * bi * Ly::RS; B = st() + 16 * bj * Ly::RS; return; }
        l -= G_X1;
        bi = l / NVB; bj = l % NVB; kind = 5; A = rows(Ly::SLOT_KN) + 16 * bi * Ly::RS; B = st() + 16 * bj * Ly::RS;
    }

    // All Gram products, K S0 products and (owned) Q S0 products of the block.
    __device__ void gram_and_x(f32x4 (&gacc)[NGW], f32x4 (&x2)[NXW], f32x4 (&x4)[NXW]) const
    {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NGW; ++s) {
            const int idx = wave + s * kWaves;
            gacc[s] = z;
            if (idx < NG) {
                int kind, bi, bj;
                const E *A, *B;
                g_decode(idx, kind, bi, bj, A, B);
                gacc[s] = tile_mma<E, DK>(z, A, Ly::RS, B, Ly::RS, lane);
            }
        }
#pragma unroll
        for (int s = 0; s < NXW; ++s) {
            const int t = wave + s * kWaves;
            x2[s] = z;
            x4[s] = z;
            if (t < NX) {
                const int bi = t / NVB, bc = t % NVB;
                if (CO) x2[s] = tile_mma<E, DK>(z, rows(Ly::SLOT_Q) + 16 * bi * Ly::RS, Ly::RS, st() + 16 * bc * Ly::RS, Ly::RS, lane);
                if (NZ) x4[s] = tile_mma<E, DK>(z, rows(Ly::SLOT_QN) + 16 * bi * Ly::RS, Ly::RS, st() + 16 * bc * Ly::RS, Ly::RS, lane);
            }
        }
    }

    // Masks, decays and beta applied to the phase-G results, written to LDS.
    __device__ void epilogue(const f32x4 (&gacc)[NGW], f32x4 (&x2)[NXW], f32x4 (&x4)[NXW]) const
    {
        const float *G = gates(GS_G), *Bt = gates(GS_B), *Gn = gates(GS_GN), *Bn = gates(GS_BN);
        const int r0 = 4 * (lane >> 4), cl = lane & 15;
#pragma unroll
        for (int s = 0; s < NGW; ++s) {
            const int idx = wave + s * kWaves;
            if (idx < NG) {
                int kind, bi, bj;
                const E *A, *B;
                g_decode(idx, kind, bi, bj, A, B);
                const f32x4 a = gacc[s];
                if (kind == 0 || kind == 2) {  // A_ri = beta_r exp(G_r - G_c) (k_r . k_c), c < r
                    const float *GG = kind == 0 ? G : Gn;
                    const float *BB = kind == 0 ? Bt : Bn;
                    float *Am = amat(kind == 0 ? MAT_C : MAT_N);
                    const int c = 16 * bj + cl;
                    const float gc = GG[c];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        Am[r * Ly::FS + c] = c < r ? BB[r] * exp2f(GG[r] - gc) * a[i] : 0.f;
                    }
                } else if (kind == 1) {        // P_rc = exp(G_r - G_c) (q_r . k_c), c <= r
                    const int c = 16 * bj + cl;
                    const float gc = G[c];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        pm()[r * Ly::TS + c] = to_e<E>(c <= r ? exp2f(G[r] - gc) * a[i] : 0.f);
                    }
                } else if (kind == 3) {        // R_rc = exp(Gn_end - Gn_c) (qn_r . kn_c)
                    const int c = 16 * bj + cl;
                    const float dc = exp2f(Gn[LP - 1] - Gn[c]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        rm()[r * Ly::TS + c] = to_e<E>(dc * a[i]);
                    }
                } else {                       // D = V - exp(G_r) (K S0)_r, stored [v][token]
                    const bool noisy = kind == 5;
                    const float *GG = noisy ? Gn : G;
                    const E *V = vs(noisy ? MAT_N : MAT_C);
                    const int vc = 16 * bj + cl;
                    const int r = 16 * bi + r0;
                    float d[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) d[i] = to_f(V[(r + i) * Ly::VS + vc]) - exp2f(GG[r + i]) * a[i];
                    st4(dmat(noisy ? MAT_N : MAT_C) + vc * Ly::TS + r, d[0], d[1], d[2], d[3]);
                }
            }
        }
#pragma unroll
        for (int s = 0; s < NXW; ++s) {
            const int t = wave + s * kWaves;
            if (t < NX) {
                const int r = 16 * (t / NVB) + r0;
                if (CO) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) x2[s][i] *= exp2f(G[r + i]);
                }
                if (NZ) {
                    const float e = exp2f(Gn[LP - 1]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) x4[s][i] *= e;
                }
            }
        }
    }

    // ----------------------------------------------------------------- UT solve
    // (I + A)^{-1} of the unit lower-triangular block matrices, in place, then
    // T = (I + A)^{-1} diag(beta) as MFMA operands.  Diagonal 16x16 blocks by forward
    // substitution (one column per lane), off-diagonal blocks row-block by row-block:
    //   X_ij = -X_ii * sum_{k=j}^{i-1} A_ik X_kj.
    __device__ void solve() const
    {
        if (wave < Ly::NSOLVE) {
            const int g = lane >> 4, j = lane & 15;
            if (g < NB) {
                float *Ab = amat(wave) + 16 * g * Ly::FS + 16 * g;
                float x[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float acc = r == j ? 1.f : 0.f;
#pragma unroll
                    for (int i = 0; i < r; ++i) acc -= Ab[r * Ly::FS + i] * x[i];
                    x[r] = acc;
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) Ab[r * Ly::FS + j] = x[r];
            }
        }
        __syncthreads();
        for (int i = 1; i < NB; ++i) {
            const int npairs = Ly::NSOLVE * i;
            for (int p = wave; p < npairs; p += kWaves) {
                const int m = p / i, j = p % i;
                const float *Am = amat(m);
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma_rr(acc, Am + 16 * i * Ly::FS + 16 * j, Ly::FS,
                                  Am + 16 * j * Ly::FS + 16 * j, Ly::FS, 16 * (i - j), lane);
                float *Y = ytmp(p);
#pragma unroll
                for (int q = 0; q < 4; ++q) Y[(4 * (lane >> 4) + q) * 16 + (lane & 15)] = acc[q];
            }
            __syncthreads();
            for (int p = wave; p < npairs; p += kWaves) {
                const int m = p / i, j = p % i;
                float *Am = amat(m);
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma_rr(acc, Am + 16 * i * Ly::FS + 16 * i, Ly::FS, ytmp(p), 16, 16, lane);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    Am[(16 * i + 4 * (lane >> 4) + q) * Ly::FS + 16 * j + (lane & 15)] = -acc[q];
            }
            __syncthreads();
        }
        // T = X diag(beta): lower triangle, zero above.
        for (int e = tid; e < Ly::NSOLVE * LP * LP; e += kThreads) {
            const int m = e / (LP * LP), rc = e % (LP * LP), r = rc / LP, c = rc % LP;
            const float *BB = gates((CL && m == MAT_C) ? GS_B : GS_BN);
            tmat(m)[r * Ly::TS + c] = to_e<E>(c <= r ? amat(m)[r * Ly::FS + c] * BB[c] : 0.f);
        }
    }

    // ----------------------------------------------------------------- phase Delta
    __device__ void deltas() const
    {
        const float *G = gates(GS_G);
        const int r0 = 4 * (lane >> 4), cl = lane & 15;
#pragma unroll
        for (int s = 0; s < NDW; ++s) {
            const int idx = wave + s * kWaves;
            if (idx < ND) {
                const bool noisy = !CL || idx >= NX;
                const int t = (CL && noisy) ? idx - NX : idx;
                const int bi = t / NVB, bc = t % NVB;
                const int m = noisy ? MAT_N : MAT_C;
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma<E, LP>(acc, tmat(m) + 16 * bi * Ly::TS, Ly::TS, dmat(m) + 16 * bc * Ly::TS, Ly::TS, lane);
                const int vc = 16 * bc + cl, r = 16 * bi + r0;
                if (noisy) {
                    st4(post(POST_N) + vc * Ly::TS + r, acc[0], acc[1], acc[2], acc[3]);
                } else {
                    st4(post(0) + vc * Ly::TS + r, acc[0], acc[1], acc[2], acc[3]);
                    const float ge = G[LP - 1];
                    st4(post(1) + vc * Ly::TS + r, exp2f(ge - G[r]) * acc[0], exp2f(ge - G[r + 1]) * acc[1],
                        exp2f(ge - G[r + 2]) * acc[2], exp2f(ge - G[r + 3]) * acc[3]);
                }
            }
        }
    }

    // ----------------------------------------------------------------- outputs
    __device__ void store_rows(Out *dst, long stride, int nvalid, int bi, int bc, f32x4 acc, float scale) const
    {
        const int r = 16 * bi + 4 * (lane >> 4), vc = 16 * bc + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (r + i < nvalid) dst[(long)(r + i) * stride + vc] = to_e<Out>(acc[i] * scale);
    }

    __device__ void outputs(const IO &io, const f32x4 (&x2)[NXW], const f32x4 (&x4)[NXW], float scale) const
    {
#pragma unroll
        for (int s = 0; s < NXW; ++s) {
            const int t = wave + s * kWaves;
            if (t < NX) {
                const int bi = t / NVB, bc = t % NVB;
                if (CO) {
                    f32x4 acc = tile_mma<E, LP>(x2[s], pm() + 16 * bi * Ly::TS, Ly::TS, post(0) + 16 * bc * Ly::TS, Ly::TS, lane);
                    store_rows(io.o, io.v_stride, io.nvalid, bi, bc, acc, scale);
                }
                if (NZ) {
                    f32x4 acc = tile_mma<E, LP>(x4[s], rm() + 16 * bi * Ly::TS, Ly::TS, post(POST_N) + 16 * bc * Ly::TS, Ly::TS, lane);
                    store_rows(io.on, io.v_stride, io.nvalid, bi, bc, acc, scale);
                }
            }
        }
    }

    // S <- gamma_n S + K^T diag(gamma_n / gamma) Delta, then refresh the S^T operand.
    __device__ void update_state(f32x4 (&S)[NSW]) const
    {
        const float decay = exp2f(gates(GS_G)[LP - 1]);
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * kWaves;
            if (t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                f32x4 acc = S[s] * decay;
                S[s] = tile_mma<E, LP>(acc, kt() + 16 * bk * Ly::TS, Ly::TS, post(1) + 16 * bc * Ly::TS, Ly::TS, lane);
            }
        }
        write_st(S);
    }

    // One block of the two-stream schedule from the state whose S^T operand is in LDS.
    __device__ void step(const IO &io, f32x4 (&S)[NSW], float scale) const
    {
        load_block(io);
        __syncthreads();
        if (CL && wave == 0) scan_gates(GS_G);
        if (NZ && wave == (CL ? 1 : 0)) scan_gates(GS_GN);
        f32x4 gacc[NGW], x2[NXW], x4[NXW];
        gram_and_x(gacc, x2, x4);
        __syncthreads();                 // row buffers are dead from here on
        epilogue(gacc, x2, x4);
        __syncthreads();
        solve();
        __syncthreads();
        deltas();
        __syncthreads();
        outputs(io, x2, x4, scale);
        if (CL) update_state(S);
        __syncthreads();
    }
};

}  // namespace bdgdn
