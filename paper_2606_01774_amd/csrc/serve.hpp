// serve.hpp -- the Diffusion-Trust serving passes over a pool of cached fp32 states
// (Appendix "Diffusion-Trust Sampling"; "Differences between the denoise pass and the
// state-update pass"), built for streaming the states from HBM: one workgroup per
// (request, v-head) unit, bf16 q/k/v, d_k = d_v = 128, blocks of up to 32 positions.
//
// For one block of n positions read from the cached state S0 (d_k x d_v), with
// block-local cumulative log-gates G_r and gamma_r = exp(G_r) (eq. per-step-fwd rewritten
// in block form; identity positions k = 0, g = 0, beta = 0 pad the block):
//   T     = (I + A)^(-1) diag(beta),  A_ri = beta_r (gamma_r / gamma_i) (k_r . k_i), i < r
//   Delta = T (V - diag(gamma) K S0)
//   denoise (block-end readout; the state is only read):
//     O~ = s [ gamma_n Q S0 + P~ Delta ],          P~_ri = (gamma_n / gamma_i) (q_r . k_i)
//   commit (token-causal; the state is advanced and written back in place):
//     O  = s [ diag(gamma) Q S0 + P Delta ],       P_ri = (gamma_r / gamma_i) (q_r . k_i), i <= r
//     S0 <- gamma_n S0 + K^T diag(gamma_n / gamma) Delta
//   commit with recorded states (the AR-Trust verify pass, Appendix "Serving-system
//   machinery", cache-and-scatter): before that, the state before each recorded position p,
//     S^(p) = gamma_(p-1) S0 + K^T diag(m_p) Delta,  m_p,j = gamma_(p-1) / gamma_j (j < p), 0 else
//   (S^(0) = S0), is written to the states buffer.
//
// Workgroup of four waves.  Each wave owns 32 columns of the state, as two 16-column
// MFMA strips interleaved by column parity: lane (g, n) holds rows 16 kb + 4g + i of
// columns 2n and 2n + 1 (of its 32), so every state row segment a wave touches is one
// 8-byte access per lane and 128 contiguous bytes per row -- the state goes from HBM
// straight into registers as MFMA operands, read once and never staged in LDS.  The
// outputs leave the accumulators the same way.  Issue order: key/query rows, gates, V,
// then the 64 KiB state; waves 0 and 1 build T and P while the state is in flight.
#pragma once

#include "ut.hpp"

namespace bdgdn {

template <typename Out, int DK, int LP, bool COMMIT, bool CO, bool REC = false>
struct Serve {
    static_assert(!REC || COMMIT, "states are recorded by the commit pass");
    typedef __bf16 In;
    typedef _Float16 E;
    typedef f16x4 QE;
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    static constexpr int NW = 4, kThreads = 64 * NW;
    static constexpr int BV = 128;              // d_v columns per workgroup
    static constexpr int NB = LP / 16, DKB = DK / 16;
    static_assert(LP == 16 || LP == 32, "blocks of up to 32 positions");
    static_assert(DK == 128, "d_k = 128");
    static constexpr bool WANT_Q = !COMMIT || CO;   // the query rows are read
    static constexpr int CPR = DK / 8;          // 16-byte chunks per row
    static constexpr int RPB = 256 / (2 * DK);  // rows per 256 bytes
    static constexpr int TS = LP + 8;           // T, P: [row][position]
    // LDS layout
    static constexpr int ROWS_B = LP * DK * 2;
    static constexpr int OFF_K = 0, OFF_Q = ROWS_B;
    static constexpr int TM_B = (LP * TS * 2 + 15) & ~15;
    static constexpr int OFF_T = 2 * ROWS_B;
    static constexpr int OFF_P = OFF_T + TM_B;
    static constexpr int OFF_FAC = OFF_P + TM_B;   // eG[64], dG[64]
    static constexpr int OFF_US = OFF_FAC + 2 * 64 * 4;   // waves 0, 1: G[64], beta[64]
    static constexpr int BYTES = OFF_US + 2 * 128 * 4;
    // row staging: 16-byte chunks of the key (and query) rows, spread over the workgroup
    static constexpr int NSETS = WANT_Q ? 2 : 1;
    static constexpr int SET_CH = LP * CPR;
    static_assert(SET_CH % kThreads == 0, "a row set spans whole staging rounds");
    static constexpr int RPS = SET_CH / kThreads;   // staging rounds per row set
    static constexpr int RPT = NSETS * RPS;

    unsigned char *smem;
    int lane, wave;

    __device__ Serve(unsigned char *s) : smem(s)
    {
        lane = threadIdx.x & 63;
        wave = wave_id();
    }

    __device__ __forceinline__ E *rows(int si) const { return reinterpret_cast<E *>(smem + (si ? OFF_Q : OFF_K)); }
    __device__ __forceinline__ E *tm(int m) const { return reinterpret_cast<E *>(smem + (m ? OFF_P : OFF_T)); }
    __device__ __forceinline__ float *fac(int m) const { return reinterpret_cast<float *>(smem + OFF_FAC) + 64 * m; }
    __device__ __forceinline__ float *us(int w) const { return reinterpret_cast<float *>(smem + OFF_US) + 128 * w; }

    // Element offset of (row, k) in a swizzled [rows][DK] matrix: chunk k/8 of a row is
    // stored at chunk (k/8) ^ (row / RPB mod CPR), which keeps the quad reads and the
    // transpose reads free of bank conflicts.
    __device__ __forceinline__ static int rofs(int row, int k)
    {
        return row * DK + ((((k >> 3) ^ ((row / RPB) & (CPR - 1))) << 3) | (k & 7));
    }
    // Bit casts through a by-value argument: applied directly to an element of an
    // ext_vector value, __builtin_bit_cast reads the vector's first element instead.
    __device__ __forceinline__ static float f_of(unsigned x) { return __builtin_bit_cast(float, x); }
    __device__ __forceinline__ static unsigned u_of(float x) { return __builtin_bit_cast(unsigned, x); }
    __device__ __forceinline__ static __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
    {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
    }

    struct Unit {
        const In *k, *q, *v;       // first row of the block (k, q: head hq; v: head h, column v0)
        const float *g, *beta;     // first row of the block (head h)
        float *state;              // the (slot, head) state, column v0
        Out *o;                    // first row of the output (head h, column v0), or null
        int qks, vst, gst;         // row strides (elements); the state rows are BV apart
        int nvalid;                // positions of the block (<= LP)
        float scale;
        float *states;             // REC: state before position nvalid - n_rec (column v0)
        int n_rec;                 // REC: recorded positions (the block's last n_rec)
        long rec_step;             // REC: elements between consecutive recorded states
    };

    // A-operand quads of K^T rows 16 kb .. 16 kb + 15 by transpose reads: lane (g, r)
    // receives K[16 rb + 4g + i][16 kb + r], i = 0..3 (the transposed-read offsets are those
    // of rofs for row 4g + (lane >> 2 & 3), columns 16 kb + 4 (lane & 3))
    __device__ __forceinline__ void kt_quads(QE (&a)[NB], int kb) const
    {
        const int g = lane >> 4;
        const int off = rofs(4 * g + ((lane >> 2) & 3), 16 * kb + 4 * (lane & 3));
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
            a[rb] = __builtin_bit_cast(QE, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                               (__attribute__((address_space(3))) s16x4 *)(rows(0) + 16 * rb * DK + off)));
    }

    // The states before the block's last n_rec positions (see the header), from the rows'
    // Delta (dl) and the cached state S of this wave's two strips; written with the same
    // 8-byte column-pair accesses as the state itself.
    __device__ void record_states(const Unit &u, const f32x4 (&S)[2][DKB], const f32x4 (&dl)[2][NB]) const
    {
        const int g = lane >> 4, n = lane & 15;
        const int c0 = 32 * wave + 2 * n;
        const float *Gs = us(0);   // cumulative log2-gates of the block (wave 0's scratch)
        QE kt[DKB][NB];
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) kt_quads(kt[kb], kb);
        f32x4 xj[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) xj[rb] = ut::ld4f(Gs + 16 * rb + 4 * g);
        const int soff = (4 * g * BV + c0) * 4;
        for (int i = 0; i < u.n_rec; ++i) {
            const int p = u.nvalid - u.n_rec + i;
            const __amdgpu_buffer_rsrc_t rs = rsrc(u.states + (long)i * u.rec_step, (unsigned)(DK * BV * 4));
            const float xp = p > 0 ? Gs[p - 1] : 0.f;
            const float gp = p > 0 ? fexp2(xp) : 1.f;
            QE uq[2][NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                f32x4 m;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int j = 16 * rb + 4 * g + e;
                    m[e] = j < p ? fexp2(-fabsf(xp - xj[rb][e])) : 0.f;
                }
                uq[0][rb] = quad_of<E>(dl[0][rb] * m);
                uq[1][rb] = quad_of<E>(dl[1][rb] * m);
            }
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                const f32x4 a = mma_q<E, NB>(S[0][kb] * gp, kt[kb], uq[0]);
                const f32x4 b = mma_q<E, NB>(S[1][kb] * gp, kt[kb], uq[1]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const u32x2 w = {u_of(a[e]), u_of(b[e])};
                    __builtin_amdgcn_raw_buffer_store_b64(w, rs, soff, (16 * kb + e) * BV * 4, 0);
                }
            }
        }
    }

    __device__ void run(const Unit &u) const
    {
        typedef const __attribute__((address_space(3))) volatile QE *LQ;
        const int tid = threadIdx.x;
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};

        // ---- issue every load: rows, gates, V, state (in the order they are needed)
        const unsigned row_bytes = (unsigned)(u.nvalid * u.qks * 2);
        const __amdgpu_buffer_rsrc_t rk = rsrc(u.k, row_bytes);
        const __amdgpu_buffer_rsrc_t rq = rsrc(u.q, row_bytes);
        u32x4 rc[RPT];
        unsigned rl[RPT];
#pragma unroll
        for (int x = 0; x < RPT; ++x) {
            const int si = x / RPS;   // compile-time: k rows, then q rows
            const int c2 = tid + kThreads * (x % RPS), t = c2 / CPR, cc = c2 % CPR;
            const unsigned go = (unsigned)(t * u.qks * 2 + cc * 16);
            rc[x] = __builtin_amdgcn_raw_buffer_load_b128(si ? rq : rk, (int)go, 0, 0);
            rl[x] = (unsigned)((si ? OFF_Q : OFF_K) + 2 * rofs(t, 8 * cc));
        }
        // (every wave loads the gates, so all waves run one straight-line load sequence and
        // the compiler's load counters stay exact; waves 0 and 1 use them)
        const unsigned gb = (unsigned)(u.nvalid * u.gst * 4);
        const int goff = (lane < LP ? lane : 0) * u.gst * 4;
        const float gv = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(u.g, gb), goff, 0, 0));
        const float bv = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(u.beta, gb), goff, 0, 0));
        const int c0 = 32 * wave + 2 * n;   // this lane's column pair within the tile
        const __amdgpu_buffer_rsrc_t rv = rsrc(u.v, (unsigned)(u.nvalid * u.vst * 2));
        unsigned vraw[NB][4];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                vraw[rb][i] = __builtin_amdgcn_raw_buffer_load_b32(rv, ((16 * rb + 4 * g + i) * u.vst + c0) * 2, 0, 0);
        // state rows 16 kb + 4g + i, columns c0, c0 + 1 (row stride BV): the lane part in
        // the vector offset, the row part a constant
        const __amdgpu_buffer_rsrc_t rs = rsrc(u.state, (unsigned)(DK * BV * 4));
        const int soff = (4 * g * BV + c0) * 4;
        u32x2 sraw[DKB][4];
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                sraw[kb][i] = __builtin_amdgcn_raw_buffer_load_b64(rs, soff, (16 * kb + i) * BV * 4, 0);

        // ---- rows to LDS as fp16
#pragma unroll
        for (int x = 0; x < RPT; ++x) {
            *reinterpret_cast<u32x4 *>(smem + rl[x]) = to_operand<In, E>(rc[x]);
        }
        lds_barrier();

        // per-lane quad offsets (row lane & 15)
        int qo[DKB];
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) qo[kb] = rofs(n, 16 * kb + 4 * g);
        auto ld_rows = [&](QE (&q)[DKB], const E *M) {
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) q[kb] = *(LQ)(M + qo[kb]);
        };

        // ---- waves 0, 1: the record (T; P and the factors) from rows and gates only
        if (wave < 2) {
            float *Gs = us(wave), *Bs = Gs + 64;
            const float x = ut::scan32(lane < LP ? gv * kLog2e : 0.f, lane);
            const float gl = ut::lane_value(x, LP - 1);
            Gs[lane] = x;
            Bs[lane] = lane < LP ? bv : 0.f;
            if (wave == 0) {
                if (lane < LP) {
                    fac(0)[lane] = fexp2(x);
                    fac(1)[lane] = fexp2(gl - x);
                }
                ut::Consts cs;
                ut::make_consts(cs, lane);
                QE kq[NB][DKB];
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) ld_rows(kq[rb], rows(0) + 16 * rb * DK);
                ut::solve_t<NB, DKB>(kq, Gs, Bs, tm(0), TS, cs, lane);
            } else if constexpr (WANT_Q) {
                // P (or P~) in the A-operand layout: with the key rows as the left factor
                // the accumulator of tile (bj, bi) is (Q K^T)^T, i.e. lane (g, n) holds
                // q_(16 bi + n) . k_(16 bj + 4g + i).
                QE kq[NB][DKB];
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) ld_rows(kq[rb], rows(0) + 16 * rb * DK);
                f32x4 gr[NB];
                float gc[NB];
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) {
                    gr[rb] = ut::ld4f(Gs + 16 * rb + 4 * g);
                    gc[rb] = Gs[16 * rb + n];
                }
#pragma unroll
                for (int bi = 0; bi < NB; ++bi) {
                    QE qq[DKB];
                    ld_rows(qq, rows(1) + 16 * bi * DK);
#pragma unroll
                    for (int bj = 0; bj < NB; ++bj) {
                        f32x4 v = z;
                        if (!COMMIT || bj <= bi) {
                            const f32x4 qk = mma_q<E, DKB>(z, kq[bj], qq);
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                // decay to the block end (denoise) or to the row (commit)
                                const float top = COMMIT ? gc[bi] : gl;
                                const bool on = !COMMIT || bj < bi || 4 * g + i <= n;
                                v[i] = on ? fexp2(-fabsf(top - gr[bj][i])) * qk[i] : 0.f;
                            }
                        }
                        st_quad(tm(1) + (16 * bi + n) * TS + 16 * bj + 4 * g, quad_of<E>(v));
                    }
                }
            }
        }

        // ---- every wave: its two strips of the state; X = K S0 and Y = Q S0
        f32x4 S[2][DKB];
        QE sq[2][DKB];
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                S[0][kb][i] = f_of(sraw[kb][i][0]);
                S[1][kb][i] = f_of(sraw[kb][i][1]);
            }
            sq[0][kb] = quad_of<E>(S[0][kb]);
            sq[1][kb] = quad_of<E>(S[1][kb]);
        }
        f32x4 X[NB][2], Y[NB][2];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[DKB];
            ld_rows(a, rows(0) + 16 * rb * DK);
            X[rb][0] = mma_q<E, DKB>(z, a, sq[0]);
            X[rb][1] = mma_q<E, DKB>(z, a, sq[1]);
            if constexpr (WANT_Q) {
                ld_rows(a, rows(1) + 16 * rb * DK);
                Y[rb][0] = mma_q<E, DKB>(z, a, sq[0]);
                Y[rb][1] = mma_q<E, DKB>(z, a, sq[1]);
            }
        }
        lds_barrier();   // T, P, factors

        // ---- Delta = T (V - diag(gamma) X)
        QE dq[2][NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            const f32x4 eg = ut::ld4f(fac(0) + 16 * rb + 4 * g);
            f32x4 d0, d1;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const unsigned w = vraw[rb][i];
                const float v0 = __builtin_bit_cast(float, w << 16), v1 = __builtin_bit_cast(float, w & 0xffff0000u);
                d0[i] = v0 - eg[i] * X[rb][0][i];
                d1[i] = v1 - eg[i] * X[rb][1][i];
            }
            dq[0][rb] = quad_of<E>(d0);
            dq[1][rb] = quad_of<E>(d1);
        }
        f32x4 dl[2][NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[NB];
            ld_quads<E, NB>(a, tm(0) + 16 * rb * TS, TS, lane);
            dl[0][rb] = mma_q<E, NB>(z, a, dq[0]);
            dl[1][rb] = mma_q<E, NB>(z, a, dq[1]);
        }

        // ---- outputs
        if constexpr (WANT_Q) {
            QE nq[2][NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                nq[0][rb] = quad_of<E>(dl[0][rb]);
                nq[1][rb] = quad_of<E>(dl[1][rb]);
            }
            const float gn = fac(0)[LP - 1];
            constexpr int SO = (int)sizeof(Out);
            const __amdgpu_buffer_rsrc_t ro = rsrc(u.o, (unsigned)(u.nvalid * u.vst * SO));
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE a[NB];
                ld_quads<E, NB>(a, tm(1) + 16 * rb * TS, TS, lane);
                f32x4 y0, y1;
                if constexpr (COMMIT) {
                    const f32x4 eg = ut::ld4f(fac(0) + 16 * rb + 4 * g);
                    y0 = Y[rb][0] * eg;
                    y1 = Y[rb][1] * eg;
                } else {
                    y0 = Y[rb][0] * gn;
                    y1 = Y[rb][1] * gn;
                }
                const f32x4 o0 = mma_q<E, NB>(y0, a, nq[0]);
                const f32x4 o1 = mma_q<E, NB>(y1, a, nq[1]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int off = ((16 * rb + 4 * g + i) * u.vst + c0) * SO;
                    if constexpr (SO == 4) {
                        const u32x2 w = {u_of(o0[i] * u.scale), u_of(o1[i] * u.scale)};
                        __builtin_amdgcn_raw_buffer_store_b64(w, ro, off, 0, 0);
                    } else {
                        const unsigned short lo = __builtin_bit_cast(unsigned short, (__bf16)(o0[i] * u.scale));
                        const unsigned short hi = __builtin_bit_cast(unsigned short, (__bf16)(o1[i] * u.scale));
                        __builtin_amdgcn_raw_buffer_store_b32((unsigned)lo | ((unsigned)hi << 16), ro, off, 0, 0);
                    }
                }
            }
        }

        // ---- commit: S0 <- gamma_n S0 + K^T diag(gamma_n / gamma) Delta, written in place
        if constexpr (COMMIT) {
            const float gn = fac(0)[LP - 1];
            if constexpr (REC) record_states(u, S, dl);
            QE uq[2][NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                const f32x4 dg = ut::ld4f(fac(1) + 16 * rb + 4 * g);
                uq[0][rb] = quad_of<E>(dl[0][rb] * dg);
                uq[1][rb] = quad_of<E>(dl[1][rb] * dg);
            }
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                QE a[NB];
                kt_quads(a, kb);
                S[0][kb] = mma_q<E, NB>(S[0][kb] * gn, a, uq[0]);
                S[1][kb] = mma_q<E, NB>(S[1][kb] * gn, a, uq[1]);
            }
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const u32x2 w = {u_of(S[0][kb][i]), u_of(S[1][kb][i])};
                    __builtin_amdgcn_raw_buffer_store_b64(w, rs, soff, (16 * kb + i) * BV * 4, 0);
                }
        }
    }
};

}  // namespace bdgdn
