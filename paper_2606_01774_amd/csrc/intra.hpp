// intra.hpp -- the block-local UT transform and masked Q K^T of the block-diffusion
// Gated Delta Rule: everything about one diffusion block that does not depend on the
// recurrent state (Appendix "Chunk-corrected values" and eq. f-blk: the WY/UT
// correction is computed from the block's keys, gates and step sizes alone).
//
// For one block of LP positions (padded with identity positions: k = 0, g = 0,
// beta = 0) and one v-head, with block-local cumulative log-gates G_r and
// gamma_r = exp(G_r):
//   A_ri  = beta_r (gamma_r / gamma_i) (k_r . k_i)      for i < r
//   T     = (I + A)^{-1} diag(beta)
//   P_ri  = (gamma_r / gamma_i) (q_r . k_i)             for i <= r   (causal, clean)
//   R_ri  = (gamma~_n / gamma~_i) (q~_r . k~_i)                      (block-end, noisy)
// and the noisy T~ from the noisy keys, gates and step sizes.  The state scan then
// needs only T, T~, P, R and the per-position factors
//   eG_r = gamma_r,  dG_r = gamma_n / gamma_r,  eGn_r = gamma~_r.
// One workgroup computes one (block, v-head) record; all records are independent.
#pragma once

#include "common.hpp"
#include "ut.hpp"

namespace bdgdn {

// Element types by input type: q/k/v rows (and the exact Gram products) keep the input
// type; the rounded intermediates T, P, R, D, Delta are fp16 for bf16 inputs (11
// significant bits instead of 8) and fp32 for fp32 inputs; with bf16 inputs the state
// and the decayed Delta enter bf16 products as hi + lo pairs.
template <typename In> struct Prec;
template <> struct Prec<__bf16> {
    typedef __bf16 Row;
    typedef _Float16 Mid;
    static constexpr bool kSplit = true;
};
template <> struct Prec<float> {
    typedef float Row;
    typedef float Mid;
    static constexpr bool kSplit = false;
};

constexpr int al16(int x) { return (x + 15) & ~15; }
constexpr int al256(int x) { return (x + 255) & ~255; }
constexpr int imax(int a, int b) { return a > b ? a : b; }

// Byte layout of one (block, v-head) record in the workspace.
template <typename Mid, int LP> struct Rec {
    static constexpr int MAT = LP * LP * (int)sizeof(Mid);   // row-major LP x LP
    static constexpr int OFF_T = 0, OFF_TN = MAT, OFF_P = 2 * MAT, OFF_R = 3 * MAT;
    static constexpr int OFF_EG = 4 * MAT;
    static constexpr int OFF_DG = OFF_EG + LP * 4;
    static constexpr int OFF_EGN = OFF_DG + LP * 4;
    static constexpr int FACT_BYTES = 3 * LP * 4;
    static constexpr int BYTES = al256(OFF_EGN + LP * 4);
};

template <typename In, int DK, int LP, int NW>
struct Intra {
    typedef typename Prec<In>::Row Row;
    typedef typename Prec<In>::Mid Mid;
    typedef Rec<Mid, LP> Rc;
    static constexpr int kThreads = 64 * NW;
    static constexpr int NB = LP / 16;
    static constexpr int NL = NB * (NB + 1) / 2;
    static constexpr int NF = NB * NB;
    // bf16 inputs: T by the register-resident doubling solve (ut::solve_t, fp16 operands),
    // which forms K K^T itself; fp32 inputs: fp32 forward substitution from A in LDS.
    static constexpr bool REG = sizeof(Mid) == 2;
    static constexpr int NG = REG ? 2 * NF : 2 * NL + 2 * NF;   // [KK lower] QK full [KnKn lower] QnKn full
    static constexpr int NGW = (NG + NW - 1) / NW;
    static constexpr int RS = DK + Mma<Row>::kPad;
    static constexpr int FS = LP + 4;
    static constexpr int EPC = 16 / (int)sizeof(Row);
    static constexpr int CPR = DK / EPC;
    static constexpr int RCH = LP * CPR;
    static constexpr int RPT = (RCH + kThreads - 1) / kThreads;
    // LDS: the four q/k row sets, then (after the Gram products) A, A~, the solve's
    // scratch and the staged T, T~, P, R in the same region.
    static constexpr int ROWS_B = al16(LP * RS * (int)sizeof(Row));
    static constexpr int A_B = al16(LP * FS * 4);
    static constexpr int OFF_A = 0;
    static constexpr int OFF_Y = 2 * A_B;
    static constexpr int Y_B = 2 * (NB > 1 ? NB - 1 : 1) * 256 * 4;
    static constexpr int OFF_STG = OFF_Y + Y_B;
    static constexpr int U_B = al16(imax(4 * ROWS_B, OFF_STG + 4 * Rc::MAT));
    static constexpr int OFF_GATES = U_B;
    static constexpr int BYTES = OFF_GATES + 4 * 64 * 4;
    static_assert(NW >= 4, "gate slots are loaded by waves 0..3");

    unsigned char *smem;
    int tid, lane, wave;

    __device__ Intra(unsigned char *s) : smem(s)
    {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = wave_id();
    }
    __device__ __forceinline__ Row *rows(int i) const { return reinterpret_cast<Row *>(smem + i * ROWS_B); }
    __device__ __forceinline__ float *amat(int m) const { return reinterpret_cast<float *>(smem + OFF_A + m * A_B); }
    __device__ __forceinline__ float *ytmp(int p) const { return reinterpret_cast<float *>(smem + OFF_Y) + p * 256; }
    __device__ __forceinline__ Mid *stg(int m) const { return reinterpret_cast<Mid *>(smem + OFF_STG + m * Rc::MAT); }
    __device__ __forceinline__ float *gates(int s) const { return reinterpret_cast<float *>(smem + OFF_GATES) + s * 64; }

    // rows: 0 = k, 1 = q, 2 = kn, 3 = qn (first row of the block, head hq); gates:
    // 0 = g, 1 = beta, 2 = gn, 3 = betan (first row, head h).  Rows at or past nvalid
    // are identity positions.
    __device__ __forceinline__ void load(const Row *const (&src)[4], long qk_stride,
                                         const float *const (&gsrc)[4], long gate_stride,
                                         int nvalid) const
    {
        const u32x4 zero = {0u, 0u, 0u, 0u};
        const int last = nvalid - 1;
        u32x4 rb[4][RPT];
#pragma unroll
        for (int s = 0; s < RPT; ++s) {
            const int c = tid + s * kThreads;
            const int cr = c < RCH ? c : RCH - 1;
            const int t = cr / CPR, cc = cr % CPR;
            const bool ok = c < RCH && t <= last;
            const long off = (long)(t <= last ? t : last) * qk_stride + cc * EPC;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const u32x4 x = *reinterpret_cast<const u32x4 *>(src[i] + off);
                rb[i][s] = ok ? x : zero;
            }
        }
        float gv = 0.f;
        if (wave < 4) {
            const float *gp = wave == 0 ? gsrc[0] : wave == 1 ? gsrc[1] : wave == 2 ? gsrc[2] : gsrc[3];
            const float x = gp[(long)(lane <= last ? lane : last) * gate_stride];
            gv = lane <= last ? x : 0.f;
        }
#pragma unroll
        for (int s = 0; s < RPT; ++s) {
            const int c = tid + s * kThreads;
            if (c < RCH) {
                const int t = c / CPR, cc = c % CPR;
#pragma unroll
                for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4 *>(rows(i) + t * RS + cc * EPC) = rb[i][s];
            }
        }
        if (wave < 4 && lane < LP) gates(wave)[lane] = gv;
    }

    // In-place inclusive scan of a gate slot, times log2 e (one wave).
    __device__ __forceinline__ void scan_gates(int slot) const
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

    // list entry -> (kind, bi, bj, A rows, B rows); kind 0 KK, 1 QK, 2 KnKn, 3 QnKn
    __device__ __forceinline__ void decode(int idx, int &kind, int &bi, int &bj) const
    {
        int l = idx;
        if constexpr (REG) {
            kind = l < NF ? 1 : 3;
            l %= NF;
            bi = l / NB;
            bj = l % NB;
            return;
        }
        if (l < NL) { kind = 0; tri_decode(l, bi, bj); return; }
        l -= NL;
        if (l < NF) { kind = 1; bi = l / NB; bj = l % NB; return; }
        l -= NF;
        if (l < NL) { kind = 2; tri_decode(l, bi, bj); return; }
        l -= NL;
        kind = 3; bi = l / NB; bj = l % NB;
    }

    __device__ __forceinline__ void gram(f32x4 (&acc)[NGW]) const
    {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NGW; ++s) {
            const int idx = wave + s * NW;
            acc[s] = z;
            if (idx < NG) {
                int kind, bi, bj;
                decode(idx, kind, bi, bj);
                const Row *A = rows(kind == 0 ? 0 : kind == 1 ? 1 : kind == 2 ? 2 : 3) + 16 * bi * RS;
                const Row *B = rows(kind <= 1 ? 0 : 2) + 16 * bj * RS;
                acc[s] = tile_mma<Row, DK>(z, A, RS, B, RS, lane);
            }
        }
    }

    // Masks, decays and beta; A (fp32) for the solve, P and R staged as Mid.
    __device__ __forceinline__ void epilogue(const f32x4 (&acc)[NGW]) const
    {
        const int r0 = 4 * (lane >> 4), cl = lane & 15;
#pragma unroll
        for (int s = 0; s < NGW; ++s) {
            const int idx = wave + s * NW;
            if (idx < NG) {
                int kind, bi, bj;
                decode(idx, kind, bi, bj);
                const f32x4 a = acc[s];
                const int c = 16 * bj + cl;
                if (kind == 0 || kind == 2) {
                    const float *GG = gates(kind == 0 ? 0 : 2), *BB = gates(kind == 0 ? 1 : 3);
                    float *Am = amat(kind == 0 ? 0 : 1);
                    const float gc = GG[c];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        Am[r * FS + c] = c < r ? BB[r] * fexp2(GG[r] - gc) * a[i] : 0.f;
                    }
                } else if (kind == 1) {
                    const float *G = gates(0);
                    const float gc = G[c];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        stg(2)[r * LP + c] = to_e<Mid>(c <= r ? fexp2(G[r] - gc) * a[i] : 0.f);
                    }
                } else {
                    const float *Gn = gates(2);
                    const float dc = fexp2(Gn[LP - 1] - Gn[c]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        stg(3)[r * LP + c] = to_e<Mid>(dc * a[i]);
                    }
                }
            }
        }
    }

    // bf16 inputs: the key rows of the wave's stream (wave 0 clean, wave 1 noisy) as fp16
    // quads (bf16 -> fp16 is exact in range), read while the row buffers are alive; then
    // T = (I + A)^(-1) diag(beta) in registers (ut::solve_t), written to the stage.
    static constexpr int DKB = DK / 16;
    typedef ut::QE QE;
    __device__ __forceinline__ void key_quads(QE (&kq)[NB][DKB]) const
    {
        const Row *K = rows(wave == 0 ? 0 : 2);
        const int r = lane & 15, c4 = 4 * (lane >> 4);
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                const Row *src = K + (16 * rb + r) * RS + 16 * kb + c4;
                kq[rb][kb] = QE{(_Float16)to_f(src[0]), (_Float16)to_f(src[1]), (_Float16)to_f(src[2]),
                                (_Float16)to_f(src[3])};
            }
    }
    __device__ __forceinline__ void solve_reg(const QE (&kq)[NB][DKB]) const
    {
        ut::Consts cs;
        ut::make_consts(cs, lane);
        ut::solve_t<NB, DKB>(kq, gates(wave == 0 ? 0 : 2), gates(wave == 0 ? 1 : 3),
                             reinterpret_cast<_Float16 *>(stg(wave)), LP, cs, lane);
    }

    // fp32 inputs: (I + A)^{-1} in place for the clean (m = 0) and noisy (m = 1) blocks, then
    // T = (I + A)^{-1} diag(beta) staged as Mid.  Diagonal 16x16 blocks by forward
    // substitution (one column per lane), then row-block by row-block:
    //   X_ij = -X_ii sum_{k=j}^{i-1} A_ik X_kj.
    __device__ __forceinline__ void solve() const
    {
        if (wave < 2) {
            const int g = lane >> 4, j = lane & 15;
            if (g < NB) {
                float *Ab = amat(wave) + 16 * g * FS + 16 * g;
                float x[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float acc = r == j ? 1.f : 0.f;
#pragma unroll
                    for (int i = 0; i < r; ++i) acc -= Ab[r * FS + i] * x[i];
                    x[r] = acc;
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) Ab[r * FS + j] = x[r];
            }
        }
        lds_barrier();
        for (int i = 1; i < NB; ++i) {
            const int npairs = 2 * i;
            for (int p = wave; p < npairs; p += NW) {
                const int m = p / i, j = p % i;
                const float *Am = amat(m);
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma_rr(acc, Am + 16 * i * FS + 16 * j, FS, Am + 16 * j * FS + 16 * j, FS,
                                  16 * (i - j), lane);
                float *Y = ytmp(p);
#pragma unroll
                for (int q = 0; q < 4; ++q) Y[(4 * (lane >> 4) + q) * 16 + (lane & 15)] = acc[q];
            }
            lds_barrier();
            for (int p = wave; p < npairs; p += NW) {
                const int m = p / i, j = p % i;
                float *Am = amat(m);
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma_rr(acc, Am + 16 * i * FS + 16 * i, FS, ytmp(p), 16, 16, lane);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    Am[(16 * i + 4 * (lane >> 4) + q) * FS + 16 * j + (lane & 15)] = -acc[q];
            }
            lds_barrier();
        }
        for (int e = tid; e < 2 * LP * LP; e += kThreads) {
            const int m = e / (LP * LP), rc = e % (LP * LP), r = rc / LP, c = rc % LP;
            const float *BB = gates(m == 0 ? 1 : 3);
            stg(m)[r * LP + c] = to_e<Mid>(c <= r ? amat(m)[r * FS + c] * BB[c] : 0.f);
        }
    }

    // Staged T, T~, P, R and the factors to the record (coalesced 16-byte stores).
    __device__ __forceinline__ void store(unsigned char *rec) const
    {
        constexpr int NCH = 4 * Rc::MAT / 16;
        const u32x4 *src = reinterpret_cast<const u32x4 *>(smem + OFF_STG);
        u32x4 *dst = reinterpret_cast<u32x4 *>(rec);
        for (int c = tid; c < NCH; c += kThreads) dst[c] = src[c];
        if (tid < LP) {
            const float *G = gates(0), *Gn = gates(2);
            float *f = reinterpret_cast<float *>(rec + Rc::OFF_EG);
            f[tid] = fexp2(G[tid]);
            f[LP + tid] = fexp2(G[LP - 1] - G[tid]);
            f[2 * LP + tid] = fexp2(Gn[tid]);
        }
    }

    __device__ __forceinline__ void run(const Row *const (&src)[4], long qk_stride,
                                        const float *const (&gsrc)[4], long gate_stride, int nvalid,
                                        unsigned char *rec) const
    {
        load(src, qk_stride, gsrc, gate_stride, nvalid);
        lds_barrier();
        if (wave == 0) scan_gates(0);
        if (wave == 1) scan_gates(2);
        f32x4 acc[NGW];
        gram(acc);
        if constexpr (REG) {
            QE kq[NB][DKB];
            if (wave < 2) key_quads(kq);
            lds_barrier();   // row buffers are dead from here on
            epilogue(acc);   // P, R to the stage
            if (wave < 2) solve_reg(kq);   // T, T~ to the stage
        } else {
            lds_barrier();   // row buffers are dead from here on
            epilogue(acc);
            lds_barrier();
            solve();
        }
        lds_barrier();
        store(rec);
    }
};

}  // namespace bdgdn
