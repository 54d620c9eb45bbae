// scan.hpp -- the sequential state scan of the block-diffusion Gated Delta Rule with
// the noisy blocks fused in (Appendix eq. chunk-state, eq. f-blk, eq. noisy-block-fwd;
// the fused two-stream schedule of "Route II": each noisy block is evaluated from the
// clean boundary state held on chip, never written out).
//
// Per block, from the clean state S0 (d_k x b_v tile of the d_k x d_v state) and the
// block's record (T, T~, P, R and the decay factors; see intra.hpp):
//   X1 = K S0, X2 = Q S0, X3 = K~ S0, X4 = Q~ S0
//   D  = V  - diag(eG)  X1,      Delta  = T  D
//   D~ = V~ - diag(eGn) X3,      Delta~ = T~ D~
//   O  = s [ diag(eG) X2 + P Delta ]
//   O~ = s [ gamma~_n X4 + R Delta~ ]
//   S  = gamma_n S0 + K^T diag(dG) Delta
// One workgroup owns one (sequence or document, v-head, d_v tile) chain and walks its
// blocks in order; the next block's inputs are fetched while the current one computes.
#pragma once

#include <type_traits>

#include "intra.hpp"

namespace bdgdn {

// Pointers of one block of one chain (row r of a tensor is base + r * stride).
template <typename In, typename Out> struct ScanIO {
    const In *k, *q, *kn, *qn;   // first row, q/k head
    const In *v, *vn;            // first row, v head, column v0
    const unsigned char *rec;    // this (block, v-head) record
    Out *o, *on;                 // first row, v head, column v0
    long qk_stride, v_stride;
    int nvalid;
};

// F16X: with bf16 inputs, stage the q/k rows as fp16 and carry the state operand and
// the decayed Delta as single fp16 operands instead of bf16 hi + lo pairs.
template <typename In, typename Out, int DK, int BV, int LP, int NW, bool F16X = false>
struct Scan {
    static constexpr bool USE_F16 = F16X && __is_same(In, __bf16);
    typedef typename std::conditional<USE_F16, _Float16, typename Prec<In>::Row>::type Row;
    typedef typename Prec<In>::Mid Mid;
    static constexpr bool SPLIT = USE_F16 ? false : Prec<In>::kSplit;
    typedef Rec<Mid, LP> Rc;
    typedef ScanIO<In, Out> IO;
    static constexpr int kThreads = 64 * NW;
    static constexpr int NB = LP / 16, NVB = BV / 16;
    static constexpr int NX = NB * NVB;          // tiles of an LP x BV product
    static constexpr int NS = (DK / 16) * NVB;   // tiles of the d_k x BV state
    static constexpr int NXW = (NX + NW - 1) / NW;
    static constexpr int NSW = (NS + NW - 1) / NW;
    static constexpr int N13 = 2 * NX, N13W = (N13 + NW - 1) / NW;   // X1 and X3 tiles
    static constexpr int ND = 2 * NX, NDW = (ND + NW - 1) / NW;      // Delta and Delta~ tiles
    static constexpr int SR = (int)sizeof(Row), SM = (int)sizeof(Mid);
    static_assert(SR == SM, "row and intermediate operands share strides");
    static constexpr int PE = Mma<Row>::kPad;
    static constexpr int RS = DK + PE;   // [token][d_k] rows and ST [v][d_k]
    static constexpr int TS = LP + PE;   // [*][token] buffers
    static constexpr int VS = BV + PE;   // staged V [token][v]
    static constexpr int EPC = 16 / SR;
    // LDS layout
    static constexpr int ROWS_B = al16(LP * RS * SR);
    static_assert(sizeof(In) == SR, "inputs are staged chunk for chunk");
    static constexpr int DT_B = al16(BV * TS * SM);
    static constexpr int NPOST = SPLIT ? 4 : 3;   // Delta, decayed Delta (hi, lo), Delta~
    static constexpr int OFF_K = 0;
    static constexpr int OFF_Y = ROWS_B;          // q, kn, qn rows; later the post buffers
    static constexpr int Y_B = al16(imax(3 * ROWS_B, NPOST * DT_B));
    static constexpr int OFF_V = OFF_Y + Y_B;
    static constexpr int V_B = al16(LP * VS * SR);
    static constexpr int OFF_T = OFF_V + 2 * V_B;  // T, T~, P, R
    static constexpr int TM_B = al16(LP * TS * SM);
    static constexpr int OFF_F = OFF_T + 4 * TM_B; // eG, dG, eGn
    static constexpr int OFF_ST = OFF_F + 3 * 64 * 4;
    static constexpr int ST_B = al16(BV * RS * SR);
    static constexpr int OFF_D = OFF_ST + (SPLIT ? 2 : 1) * ST_B;
    static constexpr int BYTES = OFF_D + 2 * DT_B;
    // fetch geometry (16-byte chunks)
    static constexpr int CPR = DK / EPC, RCH = LP * CPR, RPT = (RCH + kThreads - 1) / kThreads;
    static constexpr int VCPR = BV / EPC, VCH = LP * VCPR, VPT = (VCH + kThreads - 1) / kThreads;
    static constexpr int MCPR = LP * SM / 16;   // chunks per record matrix row
    static constexpr int MCH = 4 * LP * MCPR, MPT = (MCH + kThreads - 1) / kThreads;
    static constexpr int FCH = Rc::FACT_BYTES / 16;
    static_assert(FCH <= kThreads, "factor chunks");
    static_assert(RCH % kThreads == 0 || RPT == 1, "row chunks");
    // a tile index w + s*NW is in range for every wave when the count divides evenly
    static constexpr bool S_EVEN = NS % NW == 0;

    unsigned char *smem;
    int tid, lane, wave;

    __device__ Scan(unsigned char *s) : smem(s)
    {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = wave_id();
    }
    __device__ __forceinline__ Row *rows(int i) const { return reinterpret_cast<Row *>(smem + i * ROWS_B); }
    __device__ __forceinline__ In *vs(int m) const { return reinterpret_cast<In *>(smem + OFF_V + m * V_B); }
    __device__ __forceinline__ Mid *tm(int m) const { return reinterpret_cast<Mid *>(smem + OFF_T + m * TM_B); }
    __device__ __forceinline__ float *fac(int m) const { return reinterpret_cast<float *>(smem + OFF_F) + m * 64; }
    __device__ __forceinline__ Row *st(int h) const { return reinterpret_cast<Row *>(smem + OFF_ST + h * ST_B); }
    __device__ __forceinline__ Mid *dm(int m) const { return reinterpret_cast<Mid *>(smem + OFF_D + m * DT_B); }
    // post buffers over the dead q / kn / qn rows
    __device__ __forceinline__ Mid *dl() const { return reinterpret_cast<Mid *>(smem + OFF_Y); }
    __device__ __forceinline__ Mid *dn() const { return reinterpret_cast<Mid *>(smem + OFF_Y + DT_B); }
    __device__ __forceinline__ Row *dd(int h) const { return reinterpret_cast<Row *>(smem + OFF_Y + (2 + h) * DT_B); }

    // ------------------------------------------------------------------ state
    __device__ __forceinline__ void load_state(f32x4 (&S)[NSW], const float *src, int dv) const
    {
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * NW;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            if ((S_EVEN || t < NS) && src) {
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
            const int t = wave + s * NW;
            if (S_EVEN || t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                float *p = dst + (long)(16 * bk + 4 * (lane >> 4)) * dv + 16 * bc + (lane & 15);
                p[0] = S[s][0];
                p[dv] = S[s][1];
                p[2 * dv] = S[s][2];
                p[3 * dv] = S[s][3];
            }
        }
    }
    // S^T operand(s) in LDS: ST[v][d_k]; with bf16 inputs as hi = bf16(S), lo = bf16(S - hi).
    __device__ __forceinline__ void write_st(const f32x4 (&S)[NSW]) const
    {
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * NW;
            if (S_EVEN || t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                const int off = (16 * bc + (lane & 15)) * RS + 16 * bk + 4 * (lane >> 4);
                if constexpr (SPLIT) {
                    float hi[4], lo[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        hi[i] = to_f(to_e<Row>(S[s][i]));
                        lo[i] = S[s][i] - hi[i];
                    }
                    st4(st(0) + off, hi[0], hi[1], hi[2], hi[3]);
                    st4(st(1) + off, lo[0], lo[1], lo[2], lo[3]);
                } else {
                    st4(st(0) + off, S[s][0], S[s][1], S[s][2], S[s][3]);
                }
            }
        }
    }

    // ------------------------------------------------------------------ loads
    // Raw loaded data; rows past the block end are zeroed when staged, so nothing
    // here waits for the loads to arrive.
    struct Fetched {
        u32x4 rb[4][RPT];
        u32x4 vb[2][VPT];
        u32x4 mb[MPT];
        u32x4 fb;
        int last;
    };

    __device__ __forceinline__ const In *row_src(const IO &io, int i) const
    {
        return i == 0 ? io.k : i == 1 ? io.q : i == 2 ? io.kn : io.qn;
    }

    // Rows at or past nvalid are read from the last valid row (in bounds); stage()
    // replaces them by zero.
    __device__ __forceinline__ void fetch(const IO &io, Fetched &f) const
    {
        const int last = io.nvalid - 1;
        f.last = last;
#pragma unroll
        for (int s = 0; s < RPT; ++s) {
            const int c = tid + s * kThreads;
            const int cr = c < RCH ? c : RCH - 1;
            const int t = cr / CPR, cc = cr % CPR;
            const long off = (long)(t <= last ? t : last) * io.qk_stride + cc * EPC;
#pragma unroll
            for (int i = 0; i < 4; ++i) f.rb[i][s] = *reinterpret_cast<const u32x4 *>(row_src(io, i) + off);
        }
#pragma unroll
        for (int s = 0; s < VPT; ++s) {
            const int c = tid + s * kThreads;
            const int cr = c < VCH ? c : VCH - 1;
            const int t = cr / VCPR, cc = cr % VCPR;
            const long off = (long)(t <= last ? t : last) * io.v_stride + cc * EPC;
            f.vb[0][s] = *reinterpret_cast<const u32x4 *>(io.v + off);
            f.vb[1][s] = *reinterpret_cast<const u32x4 *>(io.vn + off);
        }
        const u32x4 *rec = reinterpret_cast<const u32x4 *>(io.rec);
#pragma unroll
        for (int s = 0; s < MPT; ++s) {
            const int c = tid + s * kThreads;
            f.mb[s] = rec[c < MCH ? c : MCH - 1];
        }
        f.fb = rec[Rc::OFF_EG / 16 + (tid < FCH ? tid : FCH - 1)];
    }

    __device__ __forceinline__ void stage(const Fetched &f) const
    {
        const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int s = 0; s < RPT; ++s) {
            const int c = tid + s * kThreads;
            if (c < RCH) {
                const int t = c / CPR, cc = c % CPR;
                const bool ok = t <= f.last;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    *reinterpret_cast<u32x4 *>(rows(i) + t * RS + cc * EPC) = ok ? to_operand<In, Row>(f.rb[i][s]) : zero;
            }
        }
#pragma unroll
        for (int s = 0; s < VPT; ++s) {
            const int c = tid + s * kThreads;
            if (c < VCH) {
                const int t = c / VCPR, cc = c % VCPR;
                const bool ok = t <= f.last;
                *reinterpret_cast<u32x4 *>(vs(0) + t * VS + cc * EPC) = ok ? f.vb[0][s] : zero;
                *reinterpret_cast<u32x4 *>(vs(1) + t * VS + cc * EPC) = ok ? f.vb[1][s] : zero;
            }
        }
#pragma unroll
        for (int s = 0; s < MPT; ++s) {
            const int c = tid + s * kThreads;
            if (c < MCH) {
                const int m = c / (LP * MCPR), rr = (c / MCPR) % LP, cc = c % MCPR;
                *reinterpret_cast<u32x4 *>(tm(m) + rr * TS + cc * (16 / SM)) = f.mb[s];
            }
        }
        if (tid < FCH) {
            // factor chunk tid covers floats 4*tid .. 4*tid+3 of [eG | dG | eGn]
            const int e = 4 * tid, m = e / LP, i = e % LP;
            *reinterpret_cast<u32x4 *>(fac(m) + i) = f.fb;
        }
    }

    // ------------------------------------------------------------------ block step
    __device__ __forceinline__ f32x4 x_tile(const Row *A, int bc) const
    {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        if constexpr (SPLIT)
            return tile_mma2<Row, DK>(z, A, RS, st(0) + 16 * bc * RS, st(1) + 16 * bc * RS, RS, lane);
        else
            return tile_mma<Row, DK>(z, A, RS, st(0) + 16 * bc * RS, RS, lane);
    }

    __device__ __forceinline__ void store_rows(Out *dst, long stride, int nvalid, int bi, int bc, f32x4 acc,
                                               float scale) const
    {
        const int r = 16 * bi + 4 * (lane >> 4), vc = 16 * bc + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (r + i < nvalid) dst[(long)(r + i) * stride + vc] = to_e<Out>(acc[i] * scale);
    }

    __device__ __forceinline__ void step(const IO &io, bool has_next, const IO &next, Fetched &f,
                                         f32x4 (&S)[NSW], float scale) const
    {
        stage(f);
        lds_barrier();
        if (has_next) fetch(next, f);
        const int r0 = 4 * (lane >> 4), cl = lane & 15;
        const float *eG = fac(0), *dG = fac(1), *eGn = fac(2);
        // X1, X3 -> D, D~ (any wave); X2, X4 kept by their owners
#pragma unroll
        for (int s = 0; s < N13W; ++s) {
            const int idx = wave + s * NW;
            if (idx < N13) {
                const bool noisy = idx >= NX;
                const int t = noisy ? idx - NX : idx, bi = t / NVB, bc = t % NVB;
                const f32x4 a = x_tile(rows(noisy ? 2 : 0) + 16 * bi * RS, bc);
                const float *E = noisy ? eGn : eG;
                const In *V = vs(noisy ? 1 : 0);
                const int r = 16 * bi + r0, vc = 16 * bc + cl;
                float d[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) d[i] = to_f(V[(r + i) * VS + vc]) - E[r + i] * a[i];
                st4(dm(noisy ? 1 : 0) + vc * TS + r, d[0], d[1], d[2], d[3]);
            }
        }
        f32x4 x2[NXW], x4[NXW];
        const float gn_end = eGn[LP - 1];
#pragma unroll
        for (int s = 0; s < NXW; ++s) {
            const int t2 = wave + s * NW;
            if (t2 < NX) {
                x2[s] = x_tile(rows(1) + 16 * (t2 / NVB) * RS, t2 % NVB);
                const int r = 16 * (t2 / NVB) + r0;
#pragma unroll
                for (int i = 0; i < 4; ++i) x2[s][i] *= eG[r + i];
            }
            // X4 tile t is owned by wave (t + NX) % NW
            const int t4 = ((wave - NX % NW) + NW) % NW + s * NW;
            if (t4 < NX) {
                x4[s] = x_tile(rows(3) + 16 * (t4 / NVB) * RS, t4 % NVB);
#pragma unroll
                for (int i = 0; i < 4; ++i) x4[s][i] *= gn_end;
            }
        }
        lds_barrier();   // q / kn / qn rows and V are dead from here on
        // Delta = T D, Delta~ = T~ D~
#pragma unroll
        for (int s = 0; s < NDW; ++s) {
            const int idx = wave + s * NW;
            if (idx < ND) {
                const bool noisy = idx >= NX;
                const int t = noisy ? idx - NX : idx, bi = t / NVB, bc = t % NVB;
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = tile_mma<Mid, LP>(acc, tm(noisy ? 1 : 0) + 16 * bi * TS, TS, dm(noisy ? 1 : 0) + 16 * bc * TS, TS,
                                        lane);
                const int vc = 16 * bc + cl, r = 16 * bi + r0;
                if (noisy) {
                    st4(dn() + vc * TS + r, acc[0], acc[1], acc[2], acc[3]);
                } else {
                    st4(dl() + vc * TS + r, acc[0], acc[1], acc[2], acc[3]);
                    float e[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) e[i] = dG[r + i] * acc[i];
                    if constexpr (SPLIT) {
                        float hi[4], lo[4];
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            hi[i] = to_f(to_e<Row>(e[i]));
                            lo[i] = e[i] - hi[i];
                        }
                        st4(dd(0) + vc * TS + r, hi[0], hi[1], hi[2], hi[3]);
                        st4(dd(1) + vc * TS + r, lo[0], lo[1], lo[2], lo[3]);
                    } else {
                        st4(dd(0) + vc * TS + r, e[0], e[1], e[2], e[3]);
                    }
                }
            }
        }
        lds_barrier();
        // outputs
#pragma unroll
        for (int s = 0; s < NXW; ++s) {
            const int t2 = wave + s * NW;
            if (t2 < NX) {
                const int bi = t2 / NVB, bc = t2 % NVB;
                const f32x4 acc = tile_mma<Mid, LP>(x2[s], tm(2) + 16 * bi * TS, TS, dl() + 16 * bc * TS, TS, lane);
                store_rows(io.o, io.v_stride, io.nvalid, bi, bc, acc, scale);
            }
            const int t4 = ((wave - NX % NW) + NW) % NW + s * NW;
            if (t4 < NX) {
                const int bi = t4 / NVB, bc = t4 % NVB;
                const f32x4 acc = tile_mma<Mid, LP>(x4[s], tm(3) + 16 * bi * TS, TS, dn() + 16 * bc * TS, TS, lane);
                store_rows(io.on, io.v_stride, io.nvalid, bi, bc, acc, scale);
            }
        }
        // S <- gamma_n S + K^T diag(dG) Delta
        const float decay = eG[LP - 1];
#pragma unroll
        for (int s = 0; s < NSW; ++s) {
            const int t = wave + s * NW;
            if (S_EVEN || t < NS) {
                const int bk = t / NVB, bc = t % NVB;
                const f32x4 acc = S[s] * decay;
                if constexpr (SPLIT)
                    S[s] = tile_mma_at2<Row, LP>(acc, rows(0) + 16 * bk, RS, dd(0) + 16 * bc * TS, dd(1) + 16 * bc * TS,
                                                 TS, lane);
                else
                    S[s] = tile_mma_at<Row, LP>(acc, rows(0) + 16 * bk, RS, dd(0) + 16 * bc * TS, TS, lane);
            }
        }
        write_st(S);
        lds_barrier();
    }
};

}  // namespace bdgdn
