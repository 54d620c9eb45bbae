// scan.hpp -- the sequential state scan of the block-diffusion Gated Delta Rule with
// the noisy blocks fused in (Appendix eq. chunk-state, eq. f-blk, eq. noisy-block-fwd;
// the fused two-stream schedule of "Route II": each noisy block is evaluated from the
// clean boundary state held on chip, never written out).
//
// Per block, from the clean state S0 (the d_k x 32 column tile of the d_k x d_v state
// this workgroup owns) and the block's record (T, T~, P, R and the decay factors; see
// intra.hpp):
//   X1 = K S0, X2 = Q S0, X3 = K~ S0, X4 = Q~ S0
//   D  = V  - diag(eG)  X1,      Delta  = T  D
//   D~ = V~ - diag(eGn) X3,      Delta~ = T~ D~
//   O  = s [ diag(eG) X2 + P Delta ]
//   O~ = s [ gamma~_n X4 + R Delta~ ]
//   S  = gamma_n S0 + K^T diag(dG) Delta
//
// One workgroup of eight waves owns one (sequence or document, v-head, 32-column tile)
// chain and walks its blocks in order.  The waves split by role, two per role, one per
// 16-column half (bc) of the tile:
//   C (waves 0, 1)  the recurrence: X1, D, Delta and the state update, with the state
//                   kept in registers (fp32, plus its operand copy) and every
//                   intermediate passed from accumulator to operand in registers;
//                   publishes Delta and the new state's operand copy through LDS;
//   N (waves 2, 3)  the noisy block: X3, X4, D~, Delta~, O~ from the published state;
//   O (waves 4, 5)  the clean outputs, one block behind: X2 while C works on a
//                   block, P Delta once C has published Delta;
//   L (waves 6, 7)  the next block's loads: global loads one block ahead, converted
//                   and staged into the other half of a double-buffered LDS set,
//                   with K also staged transposed for the update.
// One workgroup barrier per block.  When two staging sets do not fit in LDS (64-position
// blocks with bf16 inputs, 32-position blocks with fp32 inputs) all eight waves stage
// each block in a phase of its own, behind a second barrier.
#pragma once

#include "intra.hpp"

namespace bdgdn {

// Operand type of the scan's MFMA products by input type: fp16 for bf16 inputs (the
// bf16 q / k rows convert exactly in fp16's normal range; the state operand, D and
// Delta keep 11 significant bits), fp32 for fp32 inputs.
template <typename In> struct ScanOp;
template <> struct ScanOp<__bf16> { typedef _Float16 type; };
template <> struct ScanOp<float> { typedef float type; };

template <typename In, typename Out, int DK, int BV, int LP>
struct Scan {
    typedef typename ScanOp<In>::type E;
    static_assert(__is_same(E, typename Prec<In>::Mid), "records hold scan operands");
    typedef Rec<E, LP> Rc;
    typedef Quad<E> QE;
    static constexpr int NW = 8, kThreads = 64 * NW;
    static constexpr int NB = LP / 16, DKB = DK / 16;
    static_assert(BV == 32, "two 16-column halves per workgroup");
    static constexpr int SE = (int)sizeof(E);
    static_assert(SE == (int)sizeof(In), "inputs are staged chunk for chunk");
    static constexpr int EPC = 16 / SE;   // elements per 16-byte chunk
    static constexpr int PE = EPC;        // row padding: 16 bytes
    static constexpr int RS = DK + PE;    // [token][d_k] rows, ST [v][d_k]
    static constexpr int TS = LP + PE;    // [*][token]: T, T~, P, R, K^T, Delta^T
    static constexpr int VS = BV + PE;    // V [token][v]
    // one staging set
    static constexpr int ROWS_B = al16(LP * RS * SE);
    // 16-bit operands read K^T straight from the K rows with LDS transpose loads; fp32
    // operands keep a staged transposed copy
    static constexpr bool TR = SE == 2;
    static constexpr int KT_B = TR ? 0 : al16(DK * TS * SE);
    static constexpr int V_B = al16(LP * VS * SE);
    static constexpr int TM_B = al16(LP * TS * SE);
    static constexpr int OFF_KT = 4 * ROWS_B;
    static constexpr int OFF_V = OFF_KT + KT_B;
    static constexpr int OFF_TM = OFF_V + 2 * V_B;
    static constexpr int OFF_FAC = OFF_TM + 4 * TM_B;
    static constexpr int SET_B = OFF_FAC + 3 * 64 * 4;
    static constexpr int ST_B = al16(BV * RS * SE);
    static constexpr int DT_B = al16(BV * TS * SE);
    static constexpr int kLds = 160 * 1024;
    static constexpr bool DBUF = 2 * SET_B + 2 * ST_B + 2 * DT_B <= kLds;
    static constexpr int NSET = DBUF ? 2 : 1;
    static constexpr int OFF_ST = NSET * SET_B;
    static constexpr int OFF_DT = OFF_ST + NSET * ST_B;
    static constexpr int BYTES = OFF_DT + 2 * DT_B;
    static_assert(BYTES <= kLds, "LDS budget");
    // the team of waves that loads and stages: L, or everyone in the single-set schedule
    static constexpr int TW = DBUF ? 2 : NW, TW0 = DBUF ? 6 : 0, TT = 64 * TW;
    static constexpr int CPR = DK / EPC;                  // chunks per q / k row
    static constexpr int KPL = 16 * CPR / 64;             // K chunks per lane and t-block
    static constexpr int NTBW = (NB + TW - 1) / TW;       // K t-blocks per team wave
    static constexpr int OPS = LP * CPR / TT;             // q, k~, q~ chunks per thread and set
    static_assert((LP * CPR) % TT == 0, "row chunks split evenly over the team");
    static constexpr int VCPR = BV / EPC;
    static constexpr int MCPR = LP / EPC, MCH = 4 * LP * MCPR;
    static constexpr int FCH = Rc::FACT_BYTES / 16;
    static_assert(FCH <= TT, "factor chunks");

    unsigned char *smem;
    int tid, lane, wave;

    __device__ Scan(unsigned char *s) : smem(s)
    {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = wave_id();
    }
    __device__ __forceinline__ unsigned char *set(int p) const { return smem + p * SET_B; }
    __device__ __forceinline__ E *rows(int p, int i) const { return reinterpret_cast<E *>(set(p) + i * ROWS_B); }
    __device__ __forceinline__ E *kt(int p) const { return reinterpret_cast<E *>(set(p) + OFF_KT); }
    __device__ __forceinline__ In *vs(int p, int m) const { return reinterpret_cast<In *>(set(p) + OFF_V + m * V_B); }
    __device__ __forceinline__ E *tm(int p, int m) const { return reinterpret_cast<E *>(set(p) + OFF_TM + m * TM_B); }
    __device__ __forceinline__ float *fac(int p, int m) const
    {
        return reinterpret_cast<float *>(set(p) + OFF_FAC) + m * 64;
    }
    __device__ __forceinline__ E *st(int b) const { return reinterpret_cast<E *>(smem + OFF_ST + b * ST_B); }
    __device__ __forceinline__ E *dt(int b) const { return reinterpret_cast<E *>(smem + OFF_DT + b * DT_B); }

    // ------------------------------------------------------------------ chain
    struct Ptrs {
        const In *k, *q, *kn, *qn, *v, *vn;   // first row of the block (v, vn: column tile)
        const unsigned char *rec;              // the block's record
        Out *o, *on;
    };
    struct Chain {
        Ptrs p0;                      // block 0
        long qk_blk, v_blk, rec_blk;  // per-block advance (elements, elements, bytes)
        int qks, vst;                 // row strides (elements)
        long len;                     // tokens
        int L;
        const float *h0;              // initial state tile (row stride dv) or null
        float *ht;                    // final state tile or null
        int dv;
        float scale;
    };
    __device__ __forceinline__ static void advance(Ptrs &p, const Chain &c)
    {
        p.k += c.qk_blk;
        p.q += c.qk_blk;
        p.kn += c.qk_blk;
        p.qn += c.qk_blk;
        p.v += c.v_blk;
        p.vn += c.v_blk;
        p.rec += c.rec_blk;
        p.o += c.v_blk;
        p.on += c.v_blk;
    }
    __device__ __forceinline__ static int nvalid_of(const Chain &c, int j)
    {
        const long rem = c.len - (long)j * c.L;
        return rem < c.L ? (int)rem : c.L;
    }

    // ------------------------------------------------------------------ loads
    // Buffer loads whose resource covers exactly the block's valid rows: rows at or
    // past the block end read as zero (identity padding), with no clamps or branches.
    // Per-lane byte offsets are fixed for the whole chain; the resources move with the
    // block.
    static constexpr int KCH = 16 * CPR;                  // K chunks per t-block
    static constexpr int VPS = LP * VCPR;                 // V chunks per stream
    static constexpr int VPL = (VPS + TT - 1) / TT;
    static_assert(MCH % TT == 0, "record chunks split evenly over the team");
    static constexpr int MPL = MCH / TT;
    struct Offs {
        unsigned k[NTBW][KPL];   // K rows of this wave's t-blocks
        unsigned o[OPS];         // q, k~, q~ rows
        unsigned v[VPL];
    };
    __device__ __forceinline__ void make_offs(const Chain &c, Offs &of) const
    {
        const int lt = tid - 64 * TW0, tw = wave - TW0;
#pragma unroll
        for (int s = 0; s < NTBW; ++s)
#pragma unroll
            for (int u = 0; u < KPL; ++u) {
                const int ch = lane + 64 * u, t = 16 * (tw + TW * s) + ch / CPR, cc = ch % CPR;
                of.k[s][u] = (unsigned)(t * c.qks * SE + cc * 16);
            }
#pragma unroll
        for (int u = 0; u < OPS; ++u) {
            const int ch = lt + TT * u, t = ch / CPR, cc = ch % CPR;
            of.o[u] = (unsigned)(t * c.qks * SE + cc * 16);
        }
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            const int ch = lt + TT * u, t = ch / VCPR, cc = ch % VCPR;
            of.v[u] = (unsigned)(t * c.vst * SE + cc * 16);
        }
    }

    struct Fetched {
        u32x4 kb[NTBW][KPL];
        u32x4 ob[3][OPS];
        u32x4 vb[2][VPL];
        u32x4 mb[MPL];
        u32x4 fb;
    };

    __device__ __forceinline__ static __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
    {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
    }
    __device__ __forceinline__ static u32x4 bload(__amdgpu_buffer_rsrc_t r, unsigned off)
    {
        return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    }

    __device__ __forceinline__ void fetch(const Ptrs &P, const Chain &c, int nvalid, const Offs &of, Fetched &f) const
    {
        const int lt = tid - 64 * TW0, tw = wave - TW0;
        const unsigned rb = (unsigned)(nvalid * c.qks * SE), vb = (unsigned)(nvalid * c.vst * SE);
        const __amdgpu_buffer_rsrc_t rk = rsrc(P.k, rb), rq = rsrc(P.q, rb), rkn = rsrc(P.kn, rb),
                                     rqn = rsrc(P.qn, rb), rv = rsrc(P.v, vb), rvn = rsrc(P.vn, vb),
                                     rr = rsrc(P.rec, (unsigned)Rc::BYTES);
#pragma unroll
        for (int s = 0; s < NTBW; ++s)
            if (tw + TW * s < NB) {
#pragma unroll
                for (int u = 0; u < KPL; ++u) f.kb[s][u] = bload(rk, of.k[s][u]);
            }
#pragma unroll
        for (int u = 0; u < OPS; ++u) {
            f.ob[0][u] = bload(rq, of.o[u]);
            f.ob[1][u] = bload(rkn, of.o[u]);
            f.ob[2][u] = bload(rqn, of.o[u]);
        }
#pragma unroll
        for (int u = 0; u < VPL; ++u)
            if (VPS % TT == 0 || lt + TT * u < VPS) {
                f.vb[0][u] = bload(rv, of.v[u]);
                f.vb[1][u] = bload(rvn, of.v[u]);
            }
#pragma unroll
        for (int u = 0; u < MPL; ++u) f.mb[u] = bload(rr, (unsigned)(16 * (lt + TT * u)));
        f.fb = bload(rr, (unsigned)(Rc::OFF_EG + 16 * (lt < FCH ? lt : 0)));
    }

    // Stage the fetched block into set p.  With NEXT, each register is refilled with the
    // matching chunk of the block at Pn right after it is written, so the next block's
    // loads are in flight for a whole block step; nvalid_n = 0 makes them read nothing.
    template <bool NEXT>
    __device__ __forceinline__ void stage_impl(int p, Fetched &f, const Ptrs &Pn, int nvalid_n, const Chain &c,
                                               const Offs &of) const
    {
        const int lt = tid - 64 * TW0, tw = wave - TW0;
        const unsigned rbn = (unsigned)(nvalid_n * c.qks * SE), vbn = (unsigned)(nvalid_n * c.vst * SE);
        const __amdgpu_buffer_rsrc_t rk = rsrc(Pn.k, rbn), rq = rsrc(Pn.q, rbn), rkn = rsrc(Pn.kn, rbn),
                                     rqn = rsrc(Pn.qn, rbn), rv = rsrc(Pn.v, vbn), rvn = rsrc(Pn.vn, vbn),
                                     rr = rsrc(Pn.rec, nvalid_n > 0 ? (unsigned)Rc::BYTES : 0u);
#pragma unroll
        for (int s = 0; s < NTBW; ++s) {
            const int tb = tw + TW * s;
            if (tb < NB) {
#pragma unroll
                for (int u = 0; u < KPL; ++u) {
                    const int ch = lane + 64 * u, t = 16 * tb + ch / CPR, cc = ch % CPR;
                    *reinterpret_cast<u32x4 *>(rows(p, 0) + t * RS + cc * EPC) = to_operand<In, E>(f.kb[s][u]);
                    if (NEXT) f.kb[s][u] = bload(rk, of.k[s][u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < OPS; ++u) {
            const int ch = lt + TT * u, t = ch / CPR, cc = ch % CPR;
#pragma unroll
            for (int si = 0; si < 3; ++si) {
                *reinterpret_cast<u32x4 *>(rows(p, 1 + si) + t * RS + cc * EPC) = to_operand<In, E>(f.ob[si][u]);
                if (NEXT) f.ob[si][u] = bload(si == 0 ? rq : si == 1 ? rkn : rqn, of.o[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            const int ch = lt + TT * u;
            if (VPS % TT == 0 || ch < VPS) {
                const int t = ch / VCPR, cc = ch % VCPR;
                *reinterpret_cast<u32x4 *>(vs(p, 0) + t * VS + cc * EPC) = f.vb[0][u];
                *reinterpret_cast<u32x4 *>(vs(p, 1) + t * VS + cc * EPC) = f.vb[1][u];
                if (NEXT) {
                    f.vb[0][u] = bload(rv, of.v[u]);
                    f.vb[1][u] = bload(rvn, of.v[u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < MPL; ++u) {
            const int ch = lt + TT * u;
            const int m = ch / (LP * MCPR), rr2 = (ch / MCPR) % LP, cc = ch % MCPR;
            *reinterpret_cast<u32x4 *>(tm(p, m) + rr2 * TS + cc * EPC) = f.mb[u];
            if (NEXT) f.mb[u] = bload(rr, (unsigned)(16 * ch));
        }
        if (lt < FCH) {
            // chunk lt holds floats 4 lt .. 4 lt + 3 of [eG | dG | eGn]
            const int e = 4 * lt, m = e / LP, i = e % LP;
            *reinterpret_cast<u32x4 *>(fac(p, m) + i) = f.fb;
        }
        if (NEXT) f.fb = bload(rr, (unsigned)(Rc::OFF_EG + 16 * (lt < FCH ? lt : 0)));
        // fp32 operands: K^T of this wave's t-blocks, from the rows it has just written
        // (LDS operations of one wave complete in order, so no barrier is needed)
#pragma unroll
        for (int s = 0; s < NTBW; ++s) {
            const int tb = tw + TW * s;
            if (!TR && tb < NB) {
#pragma unroll
                for (int u = 0; u < DK / 16; ++u) {
                    const int qd = lane + 64 * u, kk = qd % DK, g4 = qd / DK;
                    const E *src = rows(p, 0) + (16 * tb + 4 * g4) * RS + kk;
                    QE v;
                    v[0] = src[0];
                    v[1] = src[RS];
                    v[2] = src[2 * RS];
                    v[3] = src[3 * RS];
                    st_quad(kt(p) + kk * TS + 16 * tb + 4 * g4, v);
                }
            }
        }
    }
    __device__ __forceinline__ void stage(int p, Fetched &f, const Chain &c, const Offs &of) const
    {
        stage_impl<false>(p, f, c.p0, 0, c, of);
    }

    // ------------------------------------------------------------------ helpers
    __device__ __forceinline__ f32x4 ld4f(const float *p) const { return *reinterpret_cast<const f32x4 *>(p); }

    // X = R S for the NB row tiles of row set R (rows(p, i)), state operand quads sq.
    __device__ __forceinline__ void x_rows(f32x4 (&x)[NB], const E *R, const QE (&sq)[DKB]) const
    {
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[DKB];
            ld_quads<E, DKB>(a, R + 16 * rb * RS, RS, lane);
            x[rb] = mma_q<E, DKB>(f32x4{0.f, 0.f, 0.f, 0.f}, a, sq);
        }
    }

    // D = V - diag(G) X (column half bc), as B-operand quads.
    __device__ __forceinline__ void d_quads(QE (&dq)[NB], const f32x4 (&x)[NB], const In *V, const float *G,
                                            int bc) const
    {
        const int g = lane >> 4, n = lane & 15;
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            const int r = 16 * rb + 4 * g;
            const f32x4 gq = ld4f(G + r);
            const In *vp = V + r * VS + 16 * bc + n;
            f32x4 d;
#pragma unroll
            for (int i = 0; i < 4; ++i) d[i] = to_f(vp[i * VS]) - gq[i] * x[rb][i];
            dq[rb] = quad_of<E>(d);
        }
    }

    // Y = M Z for a record matrix M (LP x LP, rows(p)) and B-operand quads zq.
    __device__ __forceinline__ void m_times(f32x4 (&y)[NB], const E *M, const QE (&zq)[NB], const f32x4 (&init)[NB]) const
    {
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[NB];
            ld_quads<E, NB>(a, M + 16 * rb * TS, TS, lane);
            y[rb] = mma_q<E, NB>(init[rb], a, zq);
        }
    }

    __device__ __forceinline__ void store_out(Out *dst, int stride, int nvalid, int bc, const f32x4 (&acc)[NB],
                                              float scale) const
    {
        const int g = lane >> 4, n = lane & 15;
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            const int r = 16 * rb + 4 * g;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (r + i < nvalid) dst[(r + i) * stride + 16 * bc + n] = to_e<Out>(acc[rb][i] * scale);
        }
    }

    __device__ __forceinline__ void write_st(int b, const QE (&sq)[DKB], int bc) const
    {
        const int g = lane >> 4, n = lane & 15;
        E *dst = st(b) + (16 * bc + n) * RS + 4 * g;
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) st_quad(dst + 16 * kb, sq[kb]);
    }

    // A-operand quads of K^T (rows 16 kb .. 16 kb + 15 of K^T, all NB t-blocks): lane
    // (g, r) gets K[16 rb + 4 g + i][16 kb + r], i = 0..3.  A 16-bit transpose load hands
    // lane i of each 16-lane group element (i & 3) of the 4-element segment addressed by
    // lane 4 j + (i >> 2) of the group, as element j; so lane 16 g + 4 j + q addresses
    // row 16 rb + 4 g + j, columns 16 kb + 4 q .. + 3 of K.
    __device__ __forceinline__ void kt_quads(QE (&a)[NB], int p, int kb) const
    {
        if constexpr (TR) {
            const E *base = rows(p, 0) + (4 * (lane >> 4) + ((lane >> 2) & 3)) * RS + 16 * kb + 4 * (lane & 3);
#pragma unroll
            for (int rb = 0; rb < NB; ++rb)
                a[rb] = __builtin_bit_cast(QE, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                   (__attribute__((address_space(3))) s16x4 *)(base + 16 * rb * RS)));
        } else {
            ld_quads<E, NB>(a, kt(p) + 16 * kb * TS, TS, lane);
        }
    }

    // ------------------------------------------------------------------ roles
    // C: one block of the recurrence for column half bc.  S (fp32) and sq (its operand
    // copy) are the state on entry and on exit; Delta^T goes to dt(db).
    __device__ __forceinline__ void c_block(int p, int db, int bc, f32x4 (&S)[DKB], QE (&sq)[DKB]) const
    {
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z[NB] = {};
        f32x4 x[NB];
        x_rows(x, rows(p, 0), sq);
        QE dq[NB];
        d_quads(dq, x, vs(p, 0), fac(p, 0), bc);
        f32x4 dl[NB];
        m_times(dl, tm(p, 0), dq, z);
        QE uq[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            st_quad(dt(db) + (16 * bc + n) * TS + 16 * rb + 4 * g, quad_of<E>(dl[rb]));
            uq[rb] = quad_of<E>(dl[rb] * ld4f(fac(p, 1) + 16 * rb + 4 * g));
        }
        const float decay = fac(p, 0)[LP - 1];
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) {
            QE a[NB];
            kt_quads(a, p, kb);
            S[kb] = mma_q<E, NB>(S[kb] * decay, a, uq);
            sq[kb] = quad_of<E>(S[kb]);
        }
    }

    // N: the noisy block for column half bc, from the state operand in st(sb).
    __device__ __forceinline__ void n_block(int p, int sb, int bc, Out *on, int stride, int nvalid,
                                            float scale) const
    {
        const f32x4 z[NB] = {};
        QE sq[DKB];
        ld_quads<E, DKB>(sq, st(sb) + 16 * bc * RS, RS, lane);
        f32x4 x3[NB], x4[NB];
        x_rows(x3, rows(p, 2), sq);
        x_rows(x4, rows(p, 3), sq);
        QE dq[NB];
        d_quads(dq, x3, vs(p, 1), fac(p, 2), bc);
        f32x4 dn[NB];
        m_times(dn, tm(p, 1), dq, z);
        QE nq[NB];
        const float gn_end = fac(p, 2)[LP - 1];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            nq[rb] = quad_of<E>(dn[rb]);
            x4[rb] *= gn_end;
        }
        f32x4 o[NB];
        m_times(o, tm(p, 3), nq, x4);
        store_out(on, stride, nvalid, bc, o, scale);
    }

    // O, first half: X2 scaled by eG and the P quads of the current block, kept until
    // Delta is published.
    __device__ __forceinline__ void o_begin(int p, int sb, int bc, f32x4 (&x2)[NB], QE (&pq)[NB][NB]) const
    {
        const int g = lane >> 4;
        QE sq[DKB];
        ld_quads<E, DKB>(sq, st(sb) + 16 * bc * RS, RS, lane);
        x_rows(x2, rows(p, 1), sq);
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            x2[rb] *= ld4f(fac(p, 0) + 16 * rb + 4 * g);
            ld_quads<E, NB>(pq[rb], tm(p, 2) + 16 * rb * TS, TS, lane);
        }
    }

    // O, second half: O = s (X2 + P Delta) with Delta^T from dt(db).
    __device__ __forceinline__ void o_end(int db, int bc, const f32x4 (&x2)[NB], const QE (&pq)[NB][NB], Out *o,
                                          int stride, int nvalid, float scale) const
    {
        QE dq[NB];
        ld_quads<E, NB>(dq, dt(db) + 16 * bc * TS, TS, lane);
        f32x4 acc[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) acc[rb] = mma_q<E, NB>(x2[rb], pq[rb], dq);
        store_out(o, stride, nvalid, bc, acc, scale);
    }

    // ------------------------------------------------------------------ the chain
    __device__ void run(const Chain &c) const
    {
        const int nb = (int)((c.len + c.L - 1) / c.L);
        const int g = lane >> 4, n = lane & 15;
        if (wave < 2) {
            // ---- C
            const int bc = wave;
            f32x4 S[DKB];
            QE sq[DKB];
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                if (c.h0) {
                    const float *src = c.h0 + (long)(16 * kb + 4 * g) * c.dv + 16 * bc + n;
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[i] = src[i * c.dv];
                }
                S[kb] = acc;
                sq[kb] = quad_of<E>(acc);
            }
            wait_global_loads();
            Fetched f;
            Offs of;
            if (!DBUF || wave >= TW0) make_offs(c, of);
            Ptrs pf = c.p0;
            if (DBUF)
                write_st(0, sq, bc);
            else if (nb > 0)
                fetch(pf, c, nvalid_of(c, 0), of, f);
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                const int p = DBUF ? (j & 1) : 0;
                if (!DBUF) {
                    stage(0, f, c, of);
                    write_st(0, sq, bc);
                    lds_barrier();
                    if (j + 1 < nb) {
                        advance(pf, c);
                        fetch(pf, c, nvalid_of(c, j + 1), of, f);
                    }
                }
                c_block(p, j & 1, bc, S, sq);
                if (DBUF) write_st((j + 1) & 1, sq, bc);
                lds_barrier();
            }
            if (c.ht) {
#pragma unroll
                for (int kb = 0; kb < DKB; ++kb) {
                    float *dst = c.ht + (long)(16 * kb + 4 * g) * c.dv + 16 * bc + n;
#pragma unroll
                    for (int i = 0; i < 4; ++i) dst[i * c.dv] = S[kb][i];
                }
            }
        } else if (wave < 4) {
            // ---- N
            const int bc = wave - 2;
            Fetched f;
            Offs of;
            if (!DBUF || wave >= TW0) make_offs(c, of);
            Ptrs pf = c.p0, pc = c.p0;
            if (!DBUF && nb > 0) fetch(pf, c, nvalid_of(c, 0), of, f);
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                const int p = DBUF ? (j & 1) : 0;
                if (!DBUF) {
                    stage(0, f, c, of);
                    lds_barrier();
                    if (j + 1 < nb) {
                        advance(pf, c);
                        fetch(pf, c, nvalid_of(c, j + 1), of, f);
                    }
                }
                n_block(p, DBUF ? (j & 1) : 0, bc, pc.on, c.vst, nvalid_of(c, j), c.scale);
                advance(pc, c);
                lds_barrier();
            }
        } else if (wave < 6) {
            // ---- O
            const int bc = wave - 4;
            Fetched f;
            Offs of;
            if (!DBUF || wave >= TW0) make_offs(c, of);
            Ptrs pf = c.p0, pc = c.p0;
            f32x4 x2[NB];
            QE pq[NB][NB];
            if (!DBUF && nb > 0) fetch(pf, c, nvalid_of(c, 0), of, f);
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                const int p = DBUF ? (j & 1) : 0;
                if (!DBUF) {
                    stage(0, f, c, of);
                    lds_barrier();
                    if (j + 1 < nb) {
                        advance(pf, c);
                        fetch(pf, c, nvalid_of(c, j + 1), of, f);
                    }
                }
                if (j > 0) {
                    o_end((j - 1) & 1, bc, x2, pq, pc.o, c.vst, nvalid_of(c, j - 1), c.scale);
                    advance(pc, c);
                }
                o_begin(p, DBUF ? (j & 1) : 0, bc, x2, pq);
                lds_barrier();
            }
            if (nb > 0) o_end((nb - 1) & 1, bc, x2, pq, pc.o, c.vst, nvalid_of(c, nb - 1), c.scale);
        } else {
            // ---- L
            Fetched f;
            Offs of;
            if (!DBUF || wave >= TW0) make_offs(c, of);
            Ptrs pf = c.p0;
            if (nb > 0) {
                fetch(pf, c, nvalid_of(c, 0), of, f);
                if (DBUF) {
                    stage(0, f, c, of);
                    advance(pf, c);
                    if (nb > 1) fetch(pf, c, nvalid_of(c, 1), of, f);
                    advance(pf, c);
                }
            }
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                if (DBUF) {
                    // stage block j + 1, load block j + 2 (pf)
                    if (j + 1 < nb) stage_impl<true>((j + 1) & 1, f, pf, j + 2 < nb ? nvalid_of(c, j + 2) : 0, c, of);
                    advance(pf, c);
                } else {
                    stage(0, f, c, of);
                    lds_barrier();
                    if (j + 1 < nb) {
                        advance(pf, c);
                        fetch(pf, c, nvalid_of(c, j + 1), of, f);
                    }
                }
                lds_barrier();
            }
        }
    }
};

}  // namespace bdgdn
