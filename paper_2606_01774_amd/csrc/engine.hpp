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
#pragma once

#include "common.hpp"

namespace bdgdn {

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
    // row-buffer slots; slot 0 is the clean K, which lives outside U because the
    // state update at the end of the block reads it
    static constexpr int SLOT_K = 0;
    static constexpr int SLOT_Q = 1;
    static constexpr int SLOT_KN = CL ? (CO ? 2 : 1) : 0;
    static constexpr int SLOT_QN = SLOT_KN + 1;
    static constexpr int NROWS_U = NROWS - (CL ? 1 : 0);   // row sets inside U

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
    static constexpr int U_B = al(mx(NROWS_U * ROWS_B, OFF_D + NSOLVE * DT_B));

    static constexpr int OFF_K = 0;                     // clean K rows (CL only)
    static constexpr int K_B = CL ? ROWS_B : 0;
    static constexpr int OFF_U = OFF_K + K_B;
    static constexpr int OFF_ST = OFF_U + U_B;
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
template <typename In, typename E, typename Out, int DK, int BV, int LP, bool CL, bool CO, bool NZ,
          int NW = 4>
struct Engine {
    static constexpr int kWaves = NW;
    static constexpr int kThreads = 64 * NW;
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

    __device__ __forceinline__ E *rows(int slot) const
    {
        if (CL && slot == Ly::SLOT_K) return reinterpret_cast<E *>(smem + Ly::OFF_K);
        return reinterpret_cast<E *>(smem + Ly::OFF_U + (slot - (CL ? 1 : 0)) * Ly::ROWS_B);
    }
    __device__ __forceinline__ float *amat(int m) const { return reinterpret_cast<float *>(smem + Ly::OFF_U + Ly::OFF_A + m * Ly::A_B); }
    __device__ __forceinline__ float *ytmp(int p) const { return reinterpret_cast<float *>(smem + Ly::OFF_U + Ly::OFF_Y) + p * 256; }
    __device__ __forceinline__ E *tmat(int m) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + Ly::OFF_T + m * Ly::TM_B); }
    __device__ __forceinline__ E *dmat(int m) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + Ly::OFF_D + m * Ly::DT_B); }
    // post-solve [v][token] buffers: 0 = Delta, 1 = decayed Delta (clean), 2 or 0 = Delta~
    __device__ __forceinline__ E *post(int i) const { return reinterpret_cast<E *>(smem + Ly::OFF_U + Ly::OFF_POST + i * Ly::DT_B); }
    __device__ __forceinline__ E *st() const { return reinterpret_cast<E *>(smem + Ly::OFF_ST); }
    __device__ __forceinline__ E *vs(int m) const { return reinterpret_cast<E *>(smem + Ly::OFF_V + m * Ly::V_B); }
    __device__ __forceinline__ E *pm() const { return reinterpret_cast<E *>(smem + Ly::OFF_PR); }
    __device__ __forceinline__ E *rm() const { return reinterpret_cast<E *>(smem + Ly::OFF_PR + (CO ? Ly::TM_B : 0)); }
    __device__ __forceinline__ float *gates(int s) const { return reinterpret_cast<float *>(smem + Ly::OFF_GATES) + s * 64; }

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
    __device__ __forceinline__ void load_state(f32x4 (&S)[NSW], const float *src, int dv) const
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
        wait_global_loads();
    }
    __device__ __forceinline__ void store_state(const f32x4 (&S)[NSW], float *dst, int dv) const
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
    __device__ __forceinline__ void write_st(const f32x4 (&S)[NSW]) const
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
    // Global -> registers (fetch) and registers -> LDS (stage) for one block: q/k rows
    // (and K transposed), the V tiles, gates.  Rows at or past nvalid are zero:
    // identity positions (k = 0, g = 0, beta = 0).  The fetch of block b+1 is issued
    // right after block b is staged so its latency hides behind block b's work.
    // Raw loaded data (rows past the block end are zeroed when staged, so nothing here
    // waits for the loads to arrive).
    struct Fetched {
        u32x4 rb[Ly::NROWS][RPT];
        u32x4 vb[Ly::NSOLVE][VPT];
        float gv;
        int last;
    };

    // Source of row set rs (a compile-time index after unrolling).
    __device__ __forceinline__ const In *row_src(const IO &io, int rs) const
    {
        if (CL && rs == Ly::SLOT_K) return io.k;
        if (CO && rs == Ly::SLOT_Q) return io.q;
        if (NZ && rs == Ly::SLOT_KN) return io.kn;
        return io.qn;
    }

    // Rows at or past nvalid are read from the last valid row (always in bounds: a
    // block has at least one row) and replaced by zero, so every load is an
    // unconditional 16-byte global load.  Wave w < 4 reads gate slot w (one row per
    // lane), so the gate pointer is uniform across the wave.
    __device__ __forceinline__ void fetch(const IO &io, Fetched &f) const
    {
        constexpr int NR = Ly::NROWS;
        static_assert(NW >= 4, "gate slots are loaded by waves 0..3");
        const int last = io.nvalid - 1;
        f.last = last;
#pragma unroll
        for (int s = 0; s < RPT; ++s) {
            const int c = tid + s * kThreads;
            const int cr = c < RCH ? c : RCH - 1;
            const int t = cr / CPR, cc = cr % CPR;
            const long off = (long)(t <= last ? t : last) * io.qk_stride + cc * EPC;
#pragma unroll
            for (int rs = 0; rs < NR; ++rs) f.rb[rs][s] = *reinterpret_cast<const u32x4 *>(row_src(io, rs) + off);
        }
#pragma unroll
        for (int s = 0; s < VPT; ++s) {
            const int c = tid + s * kThreads;
            const int cr = c < VCH ? c : VCH - 1;
            const int t = cr / VCPR, cc = cr % VCPR;
            const long off = (long)(t <= last ? t : last) * io.v_stride + cc * EPC;
#pragma unroll
            for (int m = 0; m < Ly::NSOLVE; ++m)
                f.vb[m][s] = *reinterpret_cast<const u32x4 *>(((CL && m == 0) ? io.v : io.vn) + off);
        }
        f.gv = 0.f;
        const bool want = (wave < 2 && CL) || (wave >= 2 && wave < 4 && NZ);
        if (want) {
            const float *gp = wave == GS_G ? io.g : wave == GS_B ? io.beta : wave == GS_GN ? io.gn : io.betan;
            f.gv = gp[(long)(lane <= last ? lane : last) * io.gate_stride];
        }
    }

    __device__ __forceinline__ void stage(const Fetched &f) const
    {
        constexpr int NR = Ly::NROWS;
        const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int rs = 0; rs < NR; ++rs)
#pragma unroll
            for (int s = 0; s < RPT; ++s) {
                const int c = tid + s * kThreads;
                if (c < RCH) {
                    const int t = c / CPR, cc = c % CPR;
                    *reinterpret_cast<u32x4 *>(rows(rs) + t * Ly::RS + cc * EPC) =
                        t <= f.last ? to_operand<In, E>(f.rb[rs][s]) : zero;
                }
            }
#pragma unroll
        for (int m = 0; m < Ly::NSOLVE; ++m)
#pragma unroll
            for (int s = 0; s < VPT; ++s) {
                const int c = tid + s * kThreads;
                if (c < VCH) {
                    const int t = c / VCPR, cc = c % VCPR;
                    *reinterpret_cast<u32x4 *>(vs(m) + t * Ly::VS + cc * EPC) =
                        t <= f.last ? to_operand<In, E>(f.vb[m][s]) : zero;
                }
            }
        if (wave < 4 && lane < LP) gates(wave)[lane] = lane <= f.last ? f.gv : 0.f;
    }

    // In-place inclusive scan of a gate slot (times log2 e), by one wave.
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

    // ----------------------------------------------------------------- phase G
    // Which operands a phase-G list entry multiplies; K = DK for all of them.
    __device__ __forceinline__ void g_decode(int idx, int &kind, int &bi, int &bj, const E *&A, const E *&B) const
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
    __device__ __forceinline__ void gram_and_x(f32x4 (&gacc)[NGW], f32x4 (&x2)[NXW], f32x4 (&x4)[NXW]) const
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
    __device__ __forceinline__ void epilogue(const f32x4 (&gacc)[NGW], f32x4 (&x2)[NXW], f32x4 (&x4)[NXW]) const
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
                        Am[r * Ly::FS + c] = c < r ? BB[r] * fexp2(GG[r] - gc) * a[i] : 0.f;
                    }
                } else if (kind == 1) {        // P_rc = exp(G_r - G_c) (q_r . k_c), c <= r
                    const int c = 16 * bj + cl;
                    const float gc = G[c];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = 16 * bi + r0 + i;
                        pm()[r * Ly::TS + c] = to_e<E>(c <= r ? fexp2(G[r] - gc) * a[i] : 0.f);
                    }
                } else if (kind == 3) {        // R_rc = exp(Gn_end - Gn_c) (qn_r . kn_c)
                    const int c = 16 * bj + cl;
                    const float dc = fexp2(Gn[LP - 1] - Gn[c]);
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
                    for (int i = 0; i < 4; ++i) d[i] = to_f(V[(r + i) * Ly::VS + vc]) - fexp2(GG[r + i]) * a[i];
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
                    for (int i = 0; i < 4; ++i) x2[s][i] *= fexp2(G[r + i]);
                }
                if (NZ) {
                    const float e = fexp2(Gn[LP - 1]);
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
    __device__ __forceinline__ void solve() const
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
        lds_barrier();
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
            lds_barrier();
            for (int p = wave; p < npairs; p += kWaves) {
                const int m = p / i, j = p % i;
                float *Am = amat(m);
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma_rr(acc, Am + 16 * i * Ly::FS + 16 * i, Ly::FS, ytmp(p), 16, 16, lane);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    Am[(16 * i + 4 * (lane >> 4) + q) * Ly::FS + 16 * j + (lane & 15)] = -acc[q];
            }
            lds_barrier();
        }
        // T = X diag(beta): lower triangle, zero above.
        for (int e = tid; e < Ly::NSOLVE * LP * LP; e += kThreads) {
            const int m = e / (LP * LP), rc = e % (LP * LP), r = rc / LP, c = rc % LP;
            const float *BB = gates((CL && m == MAT_C) ? GS_B : GS_BN);
            tmat(m)[r * Ly::TS + c] = to_e<E>(c <= r ? amat(m)[r * Ly::FS + c] * BB[c] : 0.f);
        }
    }

    // ----------------------------------------------------------------- phase Delta
    __device__ __forceinline__ void deltas() const
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
                    st4(post(1) + vc * Ly::TS + r, fexp2(ge - G[r]) * acc[0], fexp2(ge - G[r + 1]) * acc[1],
                        fexp2(ge - G[r + 2]) * acc[2], fexp2(ge - G[r + 3]) * acc[3]);
                }
            }
        }
    }

    // ----------------------------------------------------------------- outputs
    __device__ __forceinline__ void store_rows(Out *dst, long stride, int nvalid, int bi, int bc, f32x4 acc, float scale) const
    {
        const int r = 16 * bi + 4 * (lane >> 4), vc = 16 * bc + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (r + i < nvalid) dst[(long)(r + i) * stride + vc] = to_e<Out>(acc[i] * scale);
    }

    __device__ __forceinline__ void outputs(const IO &io, const f32x4 (&x2)[NXW], const f32x4 (&x4)[NXW], float scale) const
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
    __device__ __forceinline__ void update_state(f32x4 (&S)[NSW]) const
    {
        const float decay = fexp2(gates(GS_G)[LP - 1]);
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * kWaves;
            if (t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                f32x4 acc = S[s] * decay;
                S[s] = tile_mma_at<E, LP>(acc, rows(Ly::SLOT_K) + 16 * bk, Ly::RS, post(1) + 16 * bc * Ly::TS, Ly::TS, lane);
            }
        }
        write_st(S);
    }

    // One block of the two-stream schedule from the state whose S^T operand is in LDS.
    // f holds this block's fetched inputs on entry; when has_next is set the inputs of
    // `next` are fetched into f while this block computes.
    __device__ __forceinline__ void step(const IO &io, bool has_next, const IO &next, Fetched &f,
                                         f32x4 (&S)[NSW], float scale) const
    {
        stage(f);
        lds_barrier();
        if (has_next) fetch(next, f);
        if (CL && wave == 0) scan_gates(GS_G);
        if (NZ && wave == (CL ? 1 : 0)) scan_gates(GS_GN);
        f32x4 gacc[NGW], x2[NXW], x4[NXW];
        gram_and_x(gacc, x2, x4);
        lds_barrier();                 // row buffers are dead from here on
        epilogue(gacc, x2, x4);
        lds_barrier();
        solve();
        lds_barrier();
        deltas();
        lds_barrier();
        outputs(io, x2, x4, scale);
        if (CL) update_state(S);
        lds_barrier();
    }
};

}  // namespace bdgdn
