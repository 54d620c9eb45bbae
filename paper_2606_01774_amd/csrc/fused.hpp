// fused.hpp -- the two-stream training forward of the block-diffusion Gated Delta Rule in
// one kernel: the block-local UT transform (Appendix "Chunk-corrected values", eq. f-blk)
// and the sequential state scan with the noisy blocks evaluated from the on-chip clean
// boundary state (Appendix eq. chunk-state, eq. noisy-block-fwd; the fused schedule of
// "Route II"), pipelined block by block inside one workgroup per (sequence or document,
// v-head, 32-column tile of d_v).
//
// Per block (see scan.hpp for the scan's arithmetic):
//   record:  G = cumulative log-gates, A_ri = beta_r 2^(G_r - G_i) (k_r . k_i) (i < r),
//            T = (I + A)^(-1) diag(beta), and the noisy T~ from the noisy rows and gates;
//   scan:    X = rows S0, D = V - diag(eG) X1, Delta = T D, O = diag(eG) Q S0 + P Delta with
//            P_ri = 2^(G_r - G_i) (q_r . k_i) (i <= r), O~ from Delta~ and
//            R_ri = 2^(G~_n - G~_i) (q~_r . k~_i), S <- gamma_n S0 + K^T diag(dG) Delta.
//
// Twelve waves in five roles; in step j of the chain
//   C (waves 0, 1)   the recurrence of block j, one 16-column half each (state in registers)
//   N (waves 2, 3)   the noisy block j, R included
//   O (waves 4, 5)   the clean outputs of block j - 1; X2 and P of block j
//   U (waves 6, 7)   the record of block j + 1: U0 the clean T and factors, U1 the noisy ones
//   L (waves 8-11)   stage the rows of block j + 2 and the V tile of block j + 1
// so nothing waits inside a step: one workgroup barrier per block.  Rows of a block live in
// a three-slot ring (used by U one step before the scan); V, the record and the factors
// in a two-slot set.  Rows are stored unpadded with their 16-byte chunks XOR-swizzled by
// row, which keeps every LDS access pattern here free of bank conflicts in 3 x 32 KB.
#pragma once

#include "intra.hpp"
#include "kernels.hpp"
#include "ut.hpp"

namespace bdgdn {

// SPLIT: the clean scan alone (the first kernel of the split schedule, Appendix "Route
// I"): the noisy waves and the noisy half of the record stand idle, the noisy rows are not
// staged, and the C waves write each block's seed state (the clean state before the
// block) to HBM for a separate noisy-block kernel.  SeedT_ is the element type of the seeds.
// STATES (with SPLIT, fp16 seeds): the recomputation of the seeds alone, for the backward:
// no clean outputs (the O waves stand idle too), and the seeds are copied from the state
// operand in LDS by the otherwise idle N waves, off the C waves' path.
// NO_O: no clean outputs (the O waves stand idle): a further noisy view of the
// complementary-view forward, whose clean stream an earlier pass has written.
// PAIR: the noisy block is two consecutive sub-blocks of the chain (blocks of 2 x the chain's
// sub-block, e.g. 64 positions as two halves of 32): the N waves carry the noisy state
// across the pair and the first half's rows also read the state at the end of the second
// (see n_block_pair).  The clean stream does not care how it is cut into blocks.
// SMALL: noisy blocks of nl positions (nl a power of two below LP, the chain's nl): the chain
// runs on LP-position clean chunks, each holding LP / nl noisy blocks whose seeds (the clean
// state at each block start inside the chunk) the N waves form from the chunk-start state
// and the chunk's clean Delta (see n_block_small).
template <typename Out, int DK, int LP, bool SPLIT = false, bool SEEDS = SPLIT, typename SeedT_ = float,
          bool STATES = false, bool NO_O = false, bool PAIR = false, bool SMALL = false>
struct Fused {
    typedef SeedT_ SeedT;
    static_assert(!STATES || (SPLIT && SEEDS && sizeof(SeedT_) == 2), "STATES: the split scan, fp16 seeds");
    typedef __bf16 In;
    typedef _Float16 E;
    typedef Quad<E> QE;
    typedef Out OutT;
    static constexpr int DKC = DK;
    static constexpr bool kSplit = SPLIT;
    static constexpr bool kSeeds = SEEDS;   // write the clean state before every block (the seeds)
    static constexpr int NW = 12, kThreads = 64 * NW;
    static constexpr int BV = 32, NVB = 2;
    static constexpr int NB = LP / 16, DKB = DK / 16;
    static_assert(LP == 16 || LP == 32, "blocks of 16 or 32 positions");
    static_assert(DK == 64 || DK == 128, "d_k of 64 or 128");
    static constexpr int CPR = DK / 8;           // 16-byte chunks per row
    static constexpr int RPB = 256 / (2 * DK);   // rows per 256 bytes (1 or 2)
    static constexpr int TS = LP + 8;            // record matrices, Delta^T: [*][token] rows
    static constexpr int VS = BV + 8;            // V [token][v]
    // LDS layout
    static constexpr int ROWS_B = LP * DK * 2;   // one row set (k, q, k~ or q~)
    static constexpr int RING_B = 4 * ROWS_B;    // one ring slot
    static constexpr int V_B = LP * VS * 2;
    static constexpr int TM_B = al16(LP * TS * 2);
    static constexpr int OFF_TM = 2 * V_B;
    static constexpr int OFF_FAC = OFF_TM + 2 * TM_B;
    // factors per position: 0 2^G, 1 2^(G_n - G), 3 G (clean, log2); 2 2^G~, 4 2^(G~_n - G~)
    // (noisy); SMALL: 5 2^(G~ at the end of the position's noisy block), 6 the clean G
    // before the position's noisy block starts (log2), G~ restarting at every noisy block
    static constexpr int NFAC = SMALL ? 7 : 5;
    static constexpr int SET_B = OFF_FAC + NFAC * 64 * 4;
    static constexpr int ST_B = BV * DK * 2;     // state operand [v][d_k], swizzled like rows
    static constexpr int DT_B = al16(BV * TS * 2);
    static constexpr int US_B = 2 * 64 * 4;      // per U wave: cumulative gates, beta
    static constexpr int OFF_SET = 3 * RING_B;
    static constexpr int OFF_ST = OFF_SET + 2 * SET_B;
    static constexpr int OFF_DT = OFF_ST + 2 * ST_B;
    static constexpr int OFF_US = OFF_DT + 2 * DT_B;
    static constexpr int OFF_SINK = OFF_US + 2 * US_B;
    // PAIR: the noisy state after the first half (fp16 operand, laid out like the state
    // operand), the first half's readout accumulators Y1 (fp32, per N wave and lane) and the
    // cross Gram tile R12 (fp16 A-operand quads [bi][bj][lane])
    static_assert(!PAIR || (LP == 32 && !SPLIT), "pairs of 32-position sub-blocks, noisy waves active");
    static_assert(!SMALL || (LP == 32 && !SPLIT && !PAIR && !NO_O), "small noisy blocks in 32-position chunks");
    // the staging team's per-lane sink for unassigned slots (none at 32-position blocks)
    static constexpr bool SINK_USED = (((LP * (DK / 8) + 255) / 256) * 256 != LP * (DK / 8)) ||
                                      ((((SPLIT ? 1 : 2) * LP * (BV / 8) + 255) / 256) * 256 != (SPLIT ? 1 : 2) * LP * (BV / 8));
    static constexpr int OFF_NS = OFF_SINK + (SINK_USED ? 64 * 16 : 0);
    static constexpr int OFF_Y1 = OFF_NS + (PAIR ? ST_B : 0);
    static constexpr int OFF_R12 = OFF_Y1 + (PAIR ? 2 * NB * 64 * 16 : 0);
    // SMALL: per record set, the raw Gram tiles of the block formed by the noisy U wave (fp32
    // accumulators in the A-operand layout): K~ K^T and Q~ K^T (tiles bj <= bi), then the
    // diagonal tiles of Q~ K~^T
    static constexpr int XT = NB * (NB + 1) / 2;
    static constexpr int XG_B = (2 * XT + NB) * 64 * 16;
    static constexpr int OFF_XG = OFF_R12 + (PAIR ? NB * NB * 64 * 8 : 0);
    // PAIR: per record set, the raw Gram tiles Q~ K~^T of the sub-block (fp16 A-operand quads),
    // formed by the noisy U wave
    static constexpr int RR_B = NB * NB * 64 * 8;
    static constexpr int OFF_RR = OFF_XG + (SMALL ? 2 * XG_B : 0);
    static constexpr int BYTES = OFF_RR + (PAIR ? 2 * RR_B : 0);
    static_assert(BYTES <= 160 * 1024, "LDS budget");
    // staging team
    static constexpr int TT = 256;
    static constexpr int NSETS = SPLIT ? 2 : 4;           // row sets staged per block
    static constexpr int OCH = LP * CPR;                  // chunks per row set
    static constexpr int OPS = (OCH + TT - 1) / TT;
    static constexpr int VCPR = BV / 8, VPS = LP * VCPR;  // V chunks per stream
    static constexpr int VPL = (2 * VPS + TT - 1) / TT;
    static_assert(VPS % 64 == 0, "a wave's V slot lies in one stream");
    static_assert(SINK_USED == (OPS * TT != OCH || VPL * TT != (SPLIT ? 1 : 2) * VPS), "sink sizing");

    unsigned char *smem;
    int tid, lane, wave;

    // Role of each hardware wave.  Wave w of the workgroup runs on SIMD w mod 4, and the
    // roles are placed so that the three waves of each SIMD carry similar work (measured
    // per-role busy cycles): SIMD 0 and 1 hold C, N and O; SIMD 2 and 3 hold U and two L.
    // `wave` below is the role index: 0-1 C, 2-3 N, 4-5 O, 6-7 U, 8-11 L.
    __device__ __forceinline__ static int role_of(int w)
    {
        return w < 2 ? w : w < 4 ? w + 6 : w < 6 ? w - 2 : w < 8 ? w : w < 10 ? w - 4 : w;
    }

    __device__ Fused(unsigned char *s) : smem(s)
    {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = role_of(wave_id());
    }

    // ------------------------------------------------------------------ layout
    __device__ __forceinline__ E *rows(int slot, int i) const
    {
        return reinterpret_cast<E *>(smem + slot * RING_B + i * ROWS_B);
    }
    __device__ __forceinline__ unsigned char *set(int p) const { return smem + OFF_SET + p * SET_B; }
    __device__ __forceinline__ In *vs(int p, int m) const { return reinterpret_cast<In *>(set(p) + m * V_B); }
    __device__ __forceinline__ E *tm(int p, int m) const { return reinterpret_cast<E *>(set(p) + OFF_TM + m * TM_B); }
    __device__ __forceinline__ float *fac(int p, int m) const
    {
        return reinterpret_cast<float *>(set(p) + OFF_FAC) + m * 64;
    }
    __device__ __forceinline__ E *st(int b) const { return reinterpret_cast<E *>(smem + OFF_ST + b * ST_B); }
    __device__ __forceinline__ E *dt(int b) const { return reinterpret_cast<E *>(smem + OFF_DT + b * DT_B); }
    __device__ __forceinline__ float *us(int u) const { return reinterpret_cast<float *>(smem + OFF_US + u * US_B); }
    __device__ __forceinline__ E *ns() const { return reinterpret_cast<E *>(smem + OFF_NS); }
    __device__ __forceinline__ f32x4 *y1(int bc) const
    {
        return reinterpret_cast<f32x4 *>(smem + OFF_Y1) + bc * NB * 64;
    }
    __device__ __forceinline__ f32x4 *xg(int p, int which, int bi, int bj) const
    {
        return reinterpret_cast<f32x4 *>(smem + OFF_XG + p * XG_B) + (which * XT + bi * (bi + 1) / 2 + bj) * 64;
    }
    __device__ __forceinline__ f32x4 *xr(int p, int b) const
    {
        return reinterpret_cast<f32x4 *>(smem + OFF_XG + p * XG_B) + (2 * XT + b) * 64;
    }
    __device__ __forceinline__ QE *rr(int p, int bi, int bj) const
    {
        return reinterpret_cast<QE *>(smem + OFF_RR + p * RR_B) + (bi * NB + bj) * 64;
    }
    __device__ __forceinline__ QE *r12(int bi, int bj) const
    {
        return reinterpret_cast<QE *>(smem + OFF_R12) + (bi * NB + bj) * 64;
    }

    // Element offset of (row, k) in a swizzled [rows][DK] matrix: chunk k/8 of a row is
    // stored at chunk (k/8) ^ (row / RPB mod CPR).
    __device__ __forceinline__ static int swz(int row) { return (row / RPB) & (CPR - 1); }
    __device__ __forceinline__ static int rofs(int row, int k)
    {
        return row * DK + ((((k >> 3) ^ swz(row)) << 3) | (k & 7));
    }

    // Per-lane offsets of the operand quads of a 16-row block (row lane & 15, k-block kb):
    // the swizzle depends on the row within the block only, so one set serves every row
    // block, row set and the state operand.
    struct QOffs {
        int q[DKB];    // quads: row lane & 15, k = 16 kb + 4 (lane >> 4)
        int t[DKB];    // transpose-load segments (see kt_quads)
    };
    __device__ __forceinline__ void make_qoffs(QOffs &o) const
    {
        const int r = lane & 15, g = lane >> 4;
        const int tr = 4 * g + ((lane >> 2) & 3), tq = lane & 3;
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) {
            o.q[kb] = rofs(r, 16 * kb + 4 * g);
            o.t[kb] = rofs(tr, 16 * kb + 4 * tq);
        }
    }
    template <int NKB>
    __device__ __forceinline__ void ld_q(QE (&q)[NKB], const E *M, const int (&off)[DKB]) const
    {
        typedef const __attribute__((address_space(3))) volatile QE *LQ;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) q[kb] = *(LQ)(M + off[kb]);
    }

    // ------------------------------------------------------------------ chain
    struct Ptrs {
        const In *k, *q, *kn, *qn, *v, *vn;
        const float *g, *beta, *gn, *betan;
        Out *o, *on;
    };
    struct Chain {
        Ptrs p0;
        long qk_blk, v_blk, g_blk;   // per-block advance (elements)
        int qks, vst, gst;           // row strides (elements)
        long len;
        int L;
        int nl;        // SMALL: positions per noisy block
        SeedT *bs;     // seed state of the chain's first block (column v0), or null
        long bs_blk;   // per-block advance of bs (elements)
        const float *h0;
        float *ht;
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
        p.g += c.g_blk;
        p.beta += c.g_blk;
        p.gn += c.g_blk;
        p.betan += c.g_blk;
        p.o += c.v_blk;
        p.on += c.v_blk;
    }
    __device__ __forceinline__ static int nvalid_of(const Chain &c, int j)
    {
        const long rem = c.len - (long)j * c.L;
        return rem <= 0 ? 0 : rem < c.L ? (int)rem : c.L;
    }
    __device__ __forceinline__ static __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
    {
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
    }

    // ------------------------------------------------------------------ L: staging
    // Every team thread runs the same straight-line sequence of slots (no branches, so
    // the compiler's load counters stay exact); an unassigned slot reloads the block's
    // first chunk and stores into a per-lane sink.  Resources cover exactly the block's
    // valid rows: rows past the block end read as zero.
    struct LOffs {
        unsigned rg[OPS], rl[OPS];   // rows: global byte offset, LDS byte offset in a row set
        unsigned vg[VPL], vl[VPL];   // V: global byte offset, LDS byte offset in a set
    };
    struct RowsF {
        u32x4 c[NSETS][OPS];
    };
    struct VF {
        u32x4 c[VPL];
    };
    __device__ __forceinline__ int v_base(int tw, int u) const { return tw * 64 + TT * u; }
    __device__ __forceinline__ void make_loffs(const Chain &c, int tw, LOffs &o) const
    {
        const int lt = 64 * tw + lane;
        const unsigned sink = (unsigned)(OFF_SINK + 16 * lane);
#pragma unroll
        for (int u = 0; u < OPS; ++u) {
            const int ch = lt + TT * u, t = ch / CPR, cc = ch % CPR;
            const bool ok = ch < OCH;
            o.rg[u] = ok ? (unsigned)(t * c.qks * 2 + cc * 16) : 0u;
            o.rl[u] = ok ? (unsigned)(2 * rofs(t, 8 * cc)) : sink;
        }
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            // slot u of team wave tw covers chunks vb .. vb + 63 of [V | V~]
            const int vb = v_base(tw, u);
            const bool ok = vb < (SPLIT ? 1 : 2) * VPS;
            const int m = vb / VPS, ch = (ok ? vb % VPS : 0) + lane, t = ch / VCPR, cc = ch % VCPR;
            o.vg[u] = ok ? (unsigned)(t * c.vst * 2 + cc * 16) : 0u;
            o.vl[u] = ok ? (unsigned)(m * V_B + (t * VS + cc * 8) * 2) : sink;
        }
    }
    struct RowRs {
        __amdgpu_buffer_rsrc_t r[4];
    };
    __device__ __forceinline__ RowRs row_rsrcs(const Ptrs &P, const Chain &c, int nvalid) const
    {
        const unsigned b = (unsigned)(nvalid * c.qks * 2);
        RowRs r;
        r.r[0] = rsrc(P.k, b);
        r.r[1] = rsrc(P.q, b);
        r.r[2] = rsrc(P.kn, b);
        r.r[3] = rsrc(P.qn, b);
        return r;
    }
    // The V stream of a slot is fixed per wave (a stream spans whole waves).
    __device__ __forceinline__ __amdgpu_buffer_rsrc_t v_rsrc(const Ptrs &P, const Chain &c, int nvalid, int tw,
                                                            int u) const
    {
        return rsrc(v_base(tw, u) >= VPS ? (const void *)P.vn : (const void *)P.v, (unsigned)(nvalid * c.vst * 2));
    }
    __device__ __forceinline__ static u32x4 bload(__amdgpu_buffer_rsrc_t r, unsigned off)
    {
        return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    }
    __device__ __forceinline__ void st16(unsigned char *base, unsigned off, u32x4 v) const
    {
        unsigned char *b = off >= (unsigned)OFF_SINK ? smem : base;
        *reinterpret_cast<u32x4 *>(b + off) = v;
    }
    __device__ __forceinline__ void fetch_rows(const Ptrs &P, const Chain &c, int nvalid, const LOffs &o, RowsF &f) const
    {
        const RowRs r = row_rsrcs(P, c, nvalid);
#pragma unroll
        for (int u = 0; u < OPS; ++u)
#pragma unroll
            for (int si = 0; si < NSETS; ++si)
                if (!((NO_O || STATES) && si == 1)) f.c[si][u] = bload(r.r[si], o.rg[u]);   // set 1 (clean q): O only
    }
    __device__ __forceinline__ void fetch_v(const Ptrs &P, const Chain &c, int nvalid, int tw, const LOffs &o, VF &f) const
    {
#pragma unroll
        for (int u = 0; u < VPL; ++u) f.c[u] = bload(v_rsrc(P, c, nvalid, tw, u), o.vg[u]);
    }
    // Stage rows into ring slot `slot` (converted to fp16), refilling from the block at Pn.
    __device__ __forceinline__ void stage_rows(int slot, RowsF &f, const Ptrs &Pn, const Chain &c, int nvalid_n,
                                               const LOffs &o) const
    {
        const RowRs r = row_rsrcs(Pn, c, nvalid_n);
#pragma unroll
        for (int u = 0; u < OPS; ++u)
#pragma unroll
            for (int si = 0; si < NSETS; ++si) {
                if ((NO_O || STATES) && si == 1) continue;   // the clean q rows are read by the O waves only
                st16(smem + slot * RING_B + si * ROWS_B, o.rl[u], to_operand<In, E>(f.c[si][u]));
                f.c[si][u] = bload(r.r[si], o.rg[u]);
            }
    }
    __device__ __forceinline__ void stage_v(int p, VF &f, const Ptrs &Pn, const Chain &c, int nvalid_n, int tw,
                                            const LOffs &o) const
    {
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            st16(set(p), o.vl[u], f.c[u]);
            f.c[u] = bload(v_rsrc(Pn, c, nvalid_n, tw, u), o.vg[u]);
        }
    }

    __device__ __forceinline__ f32x4 ld4f(const float *p) const { return *reinterpret_cast<const f32x4 *>(p); }

    // ------------------------------------------------------------------ U: the record
    // One U wave builds the clean (STREAM 0: T, P, eG, dG) or noisy (STREAM 1: T~, R,
    // eGn) half of the record of one block from the rows in ring slot `slot` and the
    // block's gates (gv, bv: lane t < LP holds position t; zero past the block end); the
    // solve itself is ut::solve_t.
    template <int STREAM>
    __device__ __forceinline__ void u_record(int slot, int p, float gv, float bv, const QOffs &qo,
                                             const ut::Consts &us_, int nl) const
    {
        float *Gs = us(STREAM), *Bs = Gs + 64;   // cumulative log2-gates, beta
        const float x = ut::scan32(lane < LP ? gv * kLog2e : 0.f, lane);
        const float gl = ut::lane_value(x, LP - 1);
        Gs[lane] = x;
        Bs[lane] = bv;
        if constexpr (SMALL) {
            // xb: the cumulative gate before the start of this position's noisy block (the
            // lane exchanges run on every lane; the selects follow them)
            const int pb = lane & (LP - 1) & ~(nl - 1);
            const float xp = __shfl(x, pb > 0 ? pb - 1 : 0, 64);
            const float xb = pb > 0 ? xp : 0.f;
            if (STREAM == 0) {
                if (lane < LP) {
                    fac(p, 0)[lane] = fexp2(x);
                    fac(p, 1)[lane] = fexp2(gl - x);
                    fac(p, 3)[lane] = x;
                    fac(p, 6)[lane] = xb;
                }
            } else {
                // noisy gates from the start of each noisy block; xe at its last position
                const float xs = x - xb;
                const float xe = __shfl(xs, pb + nl - 1, 64);
                if (lane < LP) {
                    fac(p, 2)[lane] = fexp2(xs);
                    fac(p, 4)[lane] = fexp2(xe - xs);
                    fac(p, 5)[lane] = fexp2(xe);
                }
            }
        } else if (lane < LP) {
            if (STREAM == 0) {
                fac(p, 0)[lane] = fexp2(x);
                fac(p, 1)[lane] = fexp2(gl - x);
                fac(p, 3)[lane] = x;
            } else {
                fac(p, 2)[lane] = fexp2(x);
                fac(p, 4)[lane] = fexp2(gl - x);
            }
        }
        const E *K = rows(slot, STREAM == 0 ? 0 : 2);
        QE kq[NB][DKB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) ld_q<DKB>(kq[rb], K + 16 * rb * DK, qo.q);
        if constexpr (SMALL && STREAM == 1) {
            ut::solve_t<NB, DKB, true, true>(kq, Gs, Bs, tm(p, 1), TS, us_, lane, nl);
            // the raw cross Gram tiles of the noisy rows with the clean keys (for the N waves a
            // step later; the clean keys sit in the same ring slot)
            const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int bj = 0; bj < NB; ++bj) {
                QE kc[DKB];
                ld_q<DKB>(kc, rows(slot, 0) + 16 * bj * DK, qo.q);
#pragma unroll
                for (int bi = bj; bi < NB; ++bi) {
                    xg(p, 0, bi, bj)[lane] = mma_q<E, DKB>(z, kc, kq[bi]);
                    QE qq[DKB];
                    ld_q<DKB>(qq, rows(slot, 3) + 16 * bi * DK, qo.q);
                    xg(p, 1, bi, bj)[lane] = mma_q<E, DKB>(z, kc, qq);
                    if (bi == bj) xr(p, bi)[lane] = mma_q<E, DKB>(z, kq[bi], qq);   // Q~ K~^T, tile (bi, bi)
                }
            }
        } else {
            ut::solve_t<NB, DKB>(kq, Gs, Bs, tm(p, STREAM == 0 ? 0 : 1), TS, us_, lane);
        }
        if constexpr (PAIR && STREAM == 1) {
            // for the N waves a step later: the raw Gram tiles Q~ K~^T of this sub-block and, when
            // it is the second half of a noisy block (odd record sets), the cross tiles
            // R12 = Q~1 K~2^T with the first half's query rows (their ring slot is still intact)
            const f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int bi = 0; bi < NB; ++bi) {
                QE qq[DKB];
                ld_q<DKB>(qq, rows(slot, 3) + 16 * bi * DK, qo.q);
#pragma unroll
                for (int bj = 0; bj < NB; ++bj) rr(p, bi, bj)[lane] = quad_of<E>(mma_q<E, DKB>(z, kq[bj], qq));
            }
            if (p == 1) {
                const int prev = slot == 0 ? 2 : slot - 1;
#pragma unroll
                for (int bi = 0; bi < NB; ++bi) {
                    QE qq[DKB];
                    ld_q<DKB>(qq, rows(prev, 3) + 16 * bi * DK, qo.q);
#pragma unroll
                    for (int bj = 0; bj < NB; ++bj) r12(bi, bj)[lane] = quad_of<E>(mma_q<E, DKB>(z, kq[bj], qq));
                }
            }
        }
    }

    // ------------------------------------------------------------------ scan helpers

    template <int NC>
    __device__ __forceinline__ void x_rows(f32x4 (&x)[NB][NC], const E *R, const QE (&sq)[NC][DKB],
                                           const QOffs &qo) const
    {
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[DKB];
            ld_q<DKB>(a, R + 16 * rb * DK, qo.q);
#pragma unroll
            for (int c = 0; c < NC; ++c) x[rb][c] = mma_q<E, DKB>(f32x4{0.f, 0.f, 0.f, 0.f}, a, sq[c]);
        }
    }
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
    // Y = M Z + init for a record matrix M (LP x LP, padded rows) and B-operand quads zq.
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
        constexpr int SO = (int)sizeof(Out);
        const __amdgpu_buffer_rsrc_t r = rsrc(dst, (unsigned)(nvalid * stride * SO));
        const int g = lane >> 4, n = lane & 15;
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int off = ((16 * rb + 4 * g + i) * stride + 16 * bc + n) * SO;
                const Out v = to_e<Out>(acc[rb][i] * scale);
                if constexpr (SO == 4)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, 0);
                else
                    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), r, off, 0, 0);
            }
    }
    __device__ __forceinline__ void write_st(int b, const QE (&sq)[DKB], int bc, const QOffs &qo) const
    {
        E *dst = st(b) + 16 * bc * DK;
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) st_quad(dst + qo.q[kb], sq[kb]);
    }
    // A-operand quads of K^T rows 16 kb .. 16 kb + 15 from the swizzled K rows with
    // transpose loads: lane 16 g + 4 j + q addresses row 16 rb + 4 g + j, columns
    // 16 kb + 4 q .. + 3, and lane (g, r) receives K[16 rb + 4 g + i][16 kb + r], i = 0..3.
    __device__ __forceinline__ void kt_quads(QE (&a)[NB], const E *K, int kb, const QOffs &qo) const
    {
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
            a[rb] = __builtin_bit_cast(QE, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                               (__attribute__((address_space(3))) s16x4 *)(K + 16 * rb * DK + qo.t[kb])));
    }

    // ------------------------------------------------------------------ scan roles
    __device__ __forceinline__ void c_block(int slot, int p, int db, int bc, f32x4 (&S)[DKB], QE (&sq)[DKB],
                                            const QOffs &qo) const
    {
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z[NB] = {};
        const QE(&sq1)[1][DKB] = *reinterpret_cast<const QE(*)[1][DKB]>(&sq);
        const E *K = rows(slot, 0);
        f32x4 x1[NB][1];
        x_rows<1>(x1, K, sq1, qo);
        f32x4 x[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) x[rb] = x1[rb][0];
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
            kt_quads(a, K, kb, qo);
            S[kb] = mma_q<E, NB>(S[kb] * decay, a, uq);
            sq[kb] = quad_of<E>(S[kb]);
        }
    }
    // N: the noisy block.  R_rc = 2^(G~_n - G~_c) (q~_r . k~_c) is formed here from the rows
    // it already holds: with the key rows as the left operand the accumulator is R^T, which
    // is the A-operand layout of R.
    __device__ __forceinline__ void n_block(int slot, int p, int sb, int bc, Out *on, int stride, int nvalid,
                                            float scale, const QOffs &qo) const
    {
        const int g = lane >> 4;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        const f32x4 zs[NB] = {};
        QE sq[DKB];
        ld_q<DKB>(sq, st(sb) + 16 * bc * DK, qo.q);
        QE kq[NB][DKB];
        f32x4 x3[NB], x4[NB];
        QE rq[NB][NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            ld_q<DKB>(kq[rb], rows(slot, 2) + 16 * rb * DK, qo.q);
            x3[rb] = mma_q<E, DKB>(z, kq[rb], sq);
        }
        const float gn_end = fac(p, 2)[LP - 1];
#pragma unroll
        for (int bi = 0; bi < NB; ++bi) {
            QE qq[DKB];
            ld_q<DKB>(qq, rows(slot, 3) + 16 * bi * DK, qo.q);
            x4[bi] = mma_q<E, DKB>(z, qq, sq) * gn_end;
#pragma unroll
            for (int bj = 0; bj < NB; ++bj)
                rq[bi][bj] = quad_of<E>(mma_q<E, DKB>(z, kq[bj], qq) * ld4f(fac(p, 4) + 16 * bj + 4 * g));
        }
        QE dq[NB];
        d_quads(dq, x3, vs(p, 1), fac(p, 2), bc);
        f32x4 dn[NB];
        m_times(dn, tm(p, 1), dq, zs);
        QE nq[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) nq[rb] = quad_of<E>(dn[rb]);
        f32x4 o[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) o[rb] = mma_q<E, NB>(x4[rb], rq[rb], nq);
        store_out(on, stride, nvalid, bc, o, scale);
    }
    // SMALL: the noisy blocks of nl positions inside one clean chunk.  Noisy block j (rows
    // p_j .. p_j + nl - 1) is seeded with the clean state before position p_j,
    //     S_(p_j) = 2^(c_j) S0 + sum_(i < p_j) 2^(c_j - G_i) k_i Delta_i^T,   c_j = G_(p_j - 1),
    // so with the chunk's clean Delta (recomputed here from its record and rows) every noisy
    // row r of block j reads
    //     X~ = diag(2^c) K~ S0 + (K~ K^T o M) Delta,   M_ri = 2^(c_r - G_i) [i < p_(j(r))],
    //     O~ = diag(gamma~_end) [diag(2^c) Q~ S0 + (Q~ K^T o M) Delta] + (R o B) Delta~,
    // with Delta~ = T~ (V~ - Gamma~ X~), the noisy gates restarting at each noisy block
    // (Gamma~, gamma~_end at the block's last position, R_rc = 2^(G~_end - G~_c) q~_r . k~_c)
    // and B, T~ block diagonal over the noisy blocks.  The Gram tiles K~ K^T, Q~ K^T (tiles
    // bj <= bi) and the diagonal tiles of R are in the A-operand layout (lane (g, n): row
    // 16 bi + n, column 16 bj + 4 g + i); the noisy U wave formed them a step earlier (raw, fp32
    // in LDS) and they are masked here.  Row quads are read from LDS where each product uses
    // them (the quad loads are not merged), which keeps the register footprint within three
    // waves per SIMD.
    __device__ __forceinline__ void n_block_small(int slot, int p, int sb, int bc, Out *on, int stride, int nvalid,
                                                  float scale, int nl, const QOffs &qo) const
    {
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        const f32x4 zs[NB] = {};
        const f16x4 zq = {};
        QE sq[DKB];
        ld_q<DKB>(sq, st(sb) + 16 * bc * DK, qo.q);
        const E *Kc = rows(slot, 0), *Kn = rows(slot, 2), *Qn = rows(slot, 3);
        // the chunk's clean Delta for this wave's 16 columns, as B-operand quads
        QE dcq[NB];
        {
            f32x4 x1[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE kc[DKB];
                ld_q<DKB>(kc, Kc + 16 * rb * DK, qo.q);
                x1[rb] = mma_q<E, DKB>(z, kc, sq);
            }
            QE dq[NB];
            d_quads(dq, x1, vs(p, 0), fac(p, 0), bc);
            f32x4 dl[NB];
            m_times(dl, tm(p, 0), dq, zs);
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) dcq[rb] = quad_of<E>(dl[rb]);
        }
        const float *Gc = fac(p, 3), *Cb = fac(p, 6);
        // M of tile (bi, bj) applied to a Gram accumulator in the A-operand layout
        auto masked = [&](f32x4 t, int bi, int bj) {
            const int r = 16 * bi + n, pj = r & ~(nl - 1);
            const float cr = Cb[r];
            const f32x4 gi = ld4f(Gc + 16 * bj + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; ++i) t[i] = 16 * bj + 4 * g + i < pj ? fexp2(-fabsf(cr - gi[i])) * t[i] : 0.f;
            return quad_of<E>(t);
        };
        // 2^c of the rows 16 rb + 4 g + i (accumulator layout)
        f32x4 ec[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            const f32x4 cb = ld4f(Cb + 16 * rb + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; ++i) ec[rb][i] = fexp2(cb[i]);
        }
        // the cross Gram tile (which: 0 K~ K^T, 1 Q~ K^T), masked
        auto cross = [&](int which, int bi, int bj) { return bj > bi ? zq : masked(xg(p, which, bi, bj)[lane], bi, bj); };
        // X~ and Delta~
        f32x4 x3[NB];
#pragma unroll
        for (int bi = 0; bi < NB; ++bi) {
            QE kq[DKB];
            ld_q<DKB>(kq, Kn + 16 * bi * DK, qo.q);
            QE mk[NB];
#pragma unroll
            for (int bj = 0; bj < NB; ++bj) mk[bj] = cross(0, bi, bj);
            x3[bi] = mma_q<E, NB>(mma_q<E, DKB>(z, kq, sq) * ec[bi], mk, dcq);
        }
        QE dq[NB];
        d_quads(dq, x3, vs(p, 1), fac(p, 2), bc);
        f32x4 dn[NB];
        m_times(dn, tm(p, 1), dq, zs);
        QE nq[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) nq[rb] = quad_of<E>(dn[rb]);
        // readout
        f32x4 o[NB];
#pragma unroll
        for (int bi = 0; bi < NB; ++bi) {
            QE qq[DKB];
            ld_q<DKB>(qq, Qn + 16 * bi * DK, qo.q);
            QE mq[NB], rq[NB];
#pragma unroll
            for (int bj = 0; bj < NB; ++bj) {
                mq[bj] = cross(1, bi, bj);
                if (bj == bi) {
                    // same noisy block: (r ^ c) < nl, within this 16 x 16 tile since nl <= 16
                    f32x4 t = xr(p, bi)[lane];
                    const f32x4 fc = ld4f(fac(p, 4) + 16 * bj + 4 * g);
#pragma unroll
                    for (int i = 0; i < 4; ++i) t[i] = ((n ^ (4 * g + i)) < nl) ? t[i] * fc[i] : 0.f;
                    rq[bj] = quad_of<E>(t);
                } else {
                    rq[bj] = zq;
                }
            }
            const f32x4 y = mma_q<E, NB>(mma_q<E, DKB>(z, qq, sq) * ec[bi], mq, dcq);
            o[bi] = mma_q<E, NB>(y * ld4f(fac(p, 5) + 16 * bi + 4 * g), rq, nq);
        }
        store_out(on, stride, nvalid, bc, o, scale);
    }
    // PAIR: one half of a noisy block of two sub-blocks.  First half (half 0), from the
    // clean seed S0: Delta~1, the readout Y1 = Q~1 S~1 of the half-end noisy state S~1 (kept
    // in LDS) and S~1 itself (the second half's seed, an fp16 operand in LDS).  Second half,
    // from S~1: its own rows as in n_block, and the first half's rows, which read the
    // block-end state too:
    //     O~1 = gamma~2 Y1 + R12 diag(2^(G~2_n - G~2_i)) Delta~2,
    // with the unscaled cross Gram tile R12 = Q~1 K~2^T, which the noisy U wave formed with
    // the second half's record.  Both halves take their R from the raw tiles Q~ K~^T of that
    // wave.  A block whose second half holds no rows stores Y1 directly.
    __device__ __forceinline__ void n_block_pair(int slot, int p, int sb, int bc, int half,
                                                 bool has_next, Out *on, Out *on_prev, int stride, int nvalid,
                                                 int nvalid_prev, float scale, const QOffs &qo) const
    {
        const int g = lane >> 4;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        const f32x4 zs[NB] = {};
        const E *seed = (half ? ns() : st(sb)) + 16 * bc * DK;
        f32x4 o[NB];
        QE uq[NB];   // Delta~ rows times the decay to the half end
        float gn_end;
        {
            QE sq[DKB];
            ld_q<DKB>(sq, seed, qo.q);
            QE kq[NB][DKB];
            f32x4 x3[NB], x4[NB];
            QE rq[NB][NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                ld_q<DKB>(kq[rb], rows(slot, 2) + 16 * rb * DK, qo.q);
                x3[rb] = mma_q<E, DKB>(z, kq[rb], sq);
            }
            gn_end = fac(p, 2)[LP - 1];
#pragma unroll
            for (int bi = 0; bi < NB; ++bi) {
                QE qq[DKB];
                ld_q<DKB>(qq, rows(slot, 3) + 16 * bi * DK, qo.q);
                x4[bi] = mma_q<E, DKB>(z, qq, sq) * gn_end;
                // R from the raw tiles the noisy U wave formed a step earlier
#pragma unroll
                for (int bj = 0; bj < NB; ++bj)
                    rq[bi][bj] = quad_of<E>(__builtin_convertvector(rr(p, bi, bj)[lane], f32x4) *
                                            ld4f(fac(p, 4) + 16 * bj + 4 * g));
            }
            QE dq[NB];
            d_quads(dq, x3, vs(p, 1), fac(p, 2), bc);
            f32x4 dn[NB];
            m_times(dn, tm(p, 1), dq, zs);
            QE nq[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                nq[rb] = quad_of<E>(dn[rb]);
                uq[rb] = quad_of<E>(dn[rb] * ld4f(fac(p, 4) + 16 * rb + 4 * g));
            }
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) o[rb] = mma_q<E, NB>(x4[rb], rq[rb], nq);
        }
        if (half == 0) {
            if (!has_next) {
                store_out(on, stride, nvalid, bc, o, scale);
                return;
            }
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) y1(bc)[rb * 64 + lane] = o[rb];
            // S~1 = gamma~ S0 + K~1^T diag(dG~) Delta~1, this wave's 16 columns
            const E *K = rows(slot, 2);
            // this wave's columns of the seed buffer; the offset is made opaque so that the
            // eight store addresses are formed here, not held in registers across the loop
            unsigned ofs = (unsigned)(OFF_NS + 32 * bc * DK);
            asm volatile("" : "+s"(ofs));
            E *dst = reinterpret_cast<E *>(smem + ofs);
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                QE a[NB];
                kt_quads(a, K, kb, qo);
                typedef const __attribute__((address_space(3))) volatile QE *LQ;
                const f32x4 s0 = __builtin_convertvector(*(LQ)(seed + qo.q[kb]), f32x4) * gn_end;
                st_quad(dst + qo.q[kb], quad_of<E>(mma_q<E, NB>(s0, a, uq)));
            }
        } else {
            store_out(on, stride, nvalid, bc, o, scale);
            f32x4 o1[NB];
#pragma unroll
            for (int bi = 0; bi < NB; ++bi) {
                QE a[NB];
#pragma unroll
                for (int bj = 0; bj < NB; ++bj) a[bj] = r12(bi, bj)[lane];
                o1[bi] = mma_q<E, NB>(y1(bc)[bi * 64 + lane] * gn_end, a, uq);
            }
            store_out(on_prev, stride, nvalid_prev, bc, o1, scale);
        }
    }
    // O, first half: X2 = diag(eG) Q S0 and P_rc = 2^(G_r - G_c) (q_r . k_c), c <= r, of
    // block j in registers (P in the A-operand layout, as for R above).
    __device__ __forceinline__ void o_begin(int slot, int p, int sb, int bc, f32x4 (&x2)[NB], QE (&pq)[NB][NB],
                                            const QOffs &qo) const
    {
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        QE sq[DKB];
        ld_q<DKB>(sq, st(sb) + 16 * bc * DK, qo.q);
        QE kq[NB][DKB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) ld_q<DKB>(kq[rb], rows(slot, 0) + 16 * rb * DK, qo.q);
        const float *G = fac(p, 3);
        f32x4 gr[NB];
        float gc[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            gr[rb] = ld4f(G + 16 * rb + 4 * g);
            gc[rb] = G[16 * rb + n];
        }
#pragma unroll
        for (int bi = 0; bi < NB; ++bi) {
            QE qq[DKB];
            ld_q<DKB>(qq, rows(slot, 1) + 16 * bi * DK, qo.q);
            x2[bi] = mma_q<E, DKB>(z, qq, sq) * ld4f(fac(p, 0) + 16 * bi + 4 * g);
#pragma unroll
            for (int bj = 0; bj < NB; ++bj) {
                f32x4 v = z;
                if (bj <= bi) {
                    const f32x4 qk = mma_q<E, DKB>(z, kq[bj], qq);   // row 16 bi + n, cols 16 bj + 4g + i
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const bool on = bj < bi || 4 * g + i <= n;
                        v[i] = on ? fexp2(-fabsf(gc[bi] - gr[bj][i])) * qk[i] : 0.f;
                    }
                }
                pq[bi][bj] = quad_of<E>(v);
            }
        }
    }
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

    // U: the record of block j + 1 in step j (block 0 before the loop); each block's gates
    // are loaded at the start of the step before the one that uses them.
    template <int STREAM>
    __device__ __forceinline__ void u_loop(const Chain &c, int nb, const QOffs &qo) const
    {
        Ptrs pg = c.p0;
        auto load_gates = [&](int jj, float &gx, float &bx) {
            const unsigned bytes = (unsigned)(nvalid_of(c, jj) * c.gst * 4);
            const __amdgpu_buffer_rsrc_t rg = rsrc(STREAM == 0 ? pg.g : pg.gn, bytes);
            const __amdgpu_buffer_rsrc_t rb = rsrc(STREAM == 0 ? pg.beta : pg.betan, bytes);
            const int off = (lane < LP ? lane : 0) * c.gst * 4;
            gx = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, off, 0, 0));
            bx = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rb, off, 0, 0));
            advance(pg, c);
        };
        ut::Consts usv;
        ut::make_consts(usv, lane);
        float gx, bx, gy, by;
        load_gates(0, gx, bx);
        load_gates(1, gy, by);
        lds_barrier();
        u_record<STREAM>(0, 0, lane < LP ? gx : 0.f, lane < LP ? bx : 0.f, qo, usv, c.nl);
        lds_barrier();
        for (int j = 0; j < nb; ++j) {
            load_gates(j + 2, gx, bx);
            u_record<STREAM>((j + 1) % 3, (j + 1) & 1, lane < LP ? gy : 0.f, lane < LP ? by : 0.f, qo, usv, c.nl);
            gy = gx;
            by = bx;
            lds_barrier();
        }
    }

    // ------------------------------------------------------------------ the chain
    // Barriers: two before the loop (rows and V of the first blocks staged; record of
    // block 0 built), then one per block.
    __device__ void run(const Chain &c) const
    {
        const int nb = (int)((c.len + c.L - 1) / c.L);
        const int g = lane >> 4, n = lane & 15;
        auto nv = [&](int jj) { return nvalid_of(c, jj); };
        QOffs qo;
        make_qoffs(qo);
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
            write_st(0, sq, bc, qo);
            lds_barrier();
            lds_barrier();
            SeedT *bs = c.bs;
            for (int j = 0; j < nb; ++j) {
                if constexpr (SEEDS && !STATES) {
                    // the seed of noisy block j: the clean state before block j
#pragma unroll
                    for (int kb = 0; kb < DKB; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            bs[(long)(16 * kb + 4 * g + i) * c.dv + 16 * bc + n] = (SeedT)S[kb][i];
                    bs += c.bs_blk;
                }
                c_block(j % 3, j & 1, j & 1, bc, S, sq, qo);
                write_st((j + 1) & 1, sq, bc, qo);
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
        } else if (STATES && wave < 4) {
            // ---- the seeds: in step j the state operand st(j & 1) holds the clean state
            // before block j (its fp16 copy, as the C waves would store it); one d_k row per
            // lane, this workgroup's BV columns as 16-byte stores
            const int a = 64 * (wave - 2) + lane;
            SeedT *bs = c.bs;
            lds_barrier();
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                const E *sv = st(j & 1);
#pragma unroll
                for (int cb = 0; cb < BV / 8; ++cb) {
                    f16x8 v8;
#pragma unroll
                    for (int e = 0; e < 8; ++e) v8[e] = sv[rofs(8 * cb + e, a)];
                    *reinterpret_cast<f16x8 *>(bs + (long)a * c.dv + 8 * cb) = v8;
                }
                bs += c.bs_blk;
                lds_barrier();
            }
        } else if (SPLIT && (wave < 4 || wave == 7 || (STATES && wave < 6))) {
            // ---- idle in the split schedule: keep the barrier count
            lds_barrier();
            lds_barrier();
            for (int j = 0; j < nb; ++j) lds_barrier();
        } else if (wave < 4) {
            // ---- N
            const int bc = wave - 2;
            Ptrs pc = c.p0;
            lds_barrier();
            lds_barrier();
            Out *on_prev = pc.on;
            for (int j = 0; j < nb; ++j) {
                if constexpr (PAIR) {
                    // chains start on block boundaries, so even sub-blocks open a block
                    const int half = j & 1;
                    n_block_pair(j % 3, half, half, bc, half, half == 0 && nv(j + 1) > 0, pc.on,
                                 on_prev, c.vst, nv(j), nv(j - 1), c.scale, qo);
                    on_prev = pc.on;
                } else if constexpr (SMALL) {
                    n_block_small(j % 3, j & 1, j & 1, bc, pc.on, c.vst, nv(j), c.scale, c.nl, qo);
                } else {
                    n_block(j % 3, j & 1, j & 1, bc, pc.on, c.vst, nv(j), c.scale, qo);
                }
                advance(pc, c);
                lds_barrier();
            }
        } else if (NO_O && wave < 6) {
            // ---- idle: no clean outputs
            lds_barrier();
            lds_barrier();
            for (int j = 0; j < nb; ++j) lds_barrier();
        } else if (wave < 6) {
            // ---- O
            const int bc = wave - 4;
            Ptrs pc = c.p0;
            f32x4 x2[NB];
            QE pq[NB][NB];
            lds_barrier();
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                if (j > 0) {
                    o_end((j - 1) & 1, bc, x2, pq, pc.o, c.vst, nv(j - 1), c.scale);
                    advance(pc, c);
                }
                o_begin(j % 3, j & 1, j & 1, bc, x2, pq, qo);
                lds_barrier();
            }
            if (nb > 0) o_end((nb - 1) & 1, bc, x2, pq, pc.o, c.vst, nv(nb - 1), c.scale);
        } else if (wave == 6) {
            u_loop<0>(c, nb, qo);
        } else if (wave == 7) {
            u_loop<1>(c, nb, qo);
        } else {
            // ---- L: step j stages the rows of block j + 2 and the V tile of block j + 1,
            // each refilled from two blocks further on
            const int tw = wave - 8;
            LOffs o;
            make_loffs(c, tw, o);
            Ptrs pr = c.p0, pv = c.p0;   // next rows / V block to load
            RowsF r0, r1;
            VF v0, v1;
            fetch_rows(pr, c, nv(0), o, r0);
            advance(pr, c);
            fetch_rows(pr, c, nv(1), o, r1);
            advance(pr, c);
            fetch_v(pv, c, nv(0), tw, o, v0);
            advance(pv, c);
            fetch_v(pv, c, nv(1), tw, o, v1);
            advance(pv, c);
            stage_rows(0, r0, pr, c, nv(2), o);   // rows 0; r0 <- rows 2
            advance(pr, c);
            stage_rows(1, r1, pr, c, nv(3), o);   // rows 1; r1 <- rows 3
            advance(pr, c);
            stage_v(0, v0, pv, c, nv(2), tw, o);   // V 0; v0 <- V 2
            advance(pv, c);
            lds_barrier();
            lds_barrier();
            // Steps in pairs with a straight-line body (a branch inside it would make the
            // compiler's load counters at the loop head wait for the newest loads); an odd
            // last step follows the loop.
            int j = 0;
            for (; j + 1 < nb; j += 2) {
                // step j: rows j + 2 (r0) into slot (j + 2) % 3, V j + 1 (v1) into set 1
                stage_rows((j + 2) % 3, r0, pr, c, nv(j + 4), o);
                advance(pr, c);
                stage_v(1, v1, pv, c, nv(j + 3), tw, o);
                advance(pv, c);
                lds_barrier();
                stage_rows((j + 3) % 3, r1, pr, c, nv(j + 5), o);
                advance(pr, c);
                stage_v(0, v0, pv, c, nv(j + 4), tw, o);
                advance(pv, c);
                lds_barrier();
            }
            if (j < nb) {
                stage_rows((j + 2) % 3, r0, pr, c, 0, o);
                stage_v(1, v1, pv, c, 0, tw, o);
                lds_barrier();
            }
        }
    }
};

// Workgroups of the chain kernels: the r = h_v / h_qk v-heads of a q/k head times the d_v
// tiles form one group of r * n_vt workgroups per (sequence, q/k head), and eight such
// groups interleave, so that the ids of one group are i, i + 8, i + 16, ...: workgroup ids
// are dealt to the eight XCDs in turn, so a group runs on one XCD and reads its q/k rows
// (shared by its v-heads and tiles) through one L2.
__host__ __device__ __forceinline__ int chain_grid(const ScanArgs &a)
{
    const int r = a.h_v / a.h_qk;
    const int n_qk = a.n_chains / r;
    return (n_qk + 7) / 8 * 8 * r * a.n_vt;
}

// One workgroup's chain: (sequence or document, v-head, d_v tile) from the block id, as
// chain_grid lays them out.
template <typename K>
__device__ __forceinline__ void run_chain(const ScanArgs &a, unsigned char *smem)
{
    static_assert(K::kThreads == 768, "launch bounds");
    typedef typename K::In In;
    typedef typename K::OutT Out;
    constexpr int DK = K::DKC;
    const int id = blockIdx.x;
    const int r = a.h_v / a.h_qk;
    const int per = 8 * r * a.n_vt;
    const int qc = (id / per) * 8 + (id % 8);   // (sequence, q/k head)
    const int wk = (id % per) / 8;             // (v-head of the group, d_v tile)
    const int vt = wk % a.n_vt;
    if (qc >= a.n_chains / r) return;
    int seq = qc / a.h_qk;
    const int h = (qc % a.h_qk) * r + wk / a.n_vt;
    if (a.n_order > 0) seq = a.order[seq];
    long base, len;
    if (a.cu) {
        base = a.cu[seq];
        len = (long)a.cu[seq + 1] - base;
    } else {
        base = (long)seq * a.T;
        len = a.T;
    }
    // seed states by global block: documents start on block boundaries, sequences own
    // ceil(T / L) blocks each
    long gblk0 = a.cu ? base / a.L : (long)seq * a.nblk;
    if constexpr (K::kSeeds) {
        if (a.seg) {   // one time segment of the chain, its seeds indexed from seg[seq]
            const long off = (long)a.blk0 * a.L, cap = (long)a.seg_len * a.L;
            len = len > off ? (len - off < cap ? len - off : cap) : 0;
            base += off;
            gblk0 = a.seg[seq];
        }
    }
    const int hq = h / (a.h_v / a.h_qk);
    const int v0 = vt * K::BV;
    typename K::Chain c;
    const long qk_off = (base * a.h_qk + hq) * DK;
    const long v_off = (base * a.h_v + h) * a.dv + v0;
    const long g_off = base * a.h_v + h;
    c.p0.k = static_cast<const In *>(a.k) + qk_off;
    c.p0.q = static_cast<const In *>(a.q) + qk_off;
    c.p0.kn = static_cast<const In *>(a.kn) + qk_off;
    c.p0.qn = static_cast<const In *>(a.qn) + qk_off;
    c.p0.v = static_cast<const In *>(a.v) + v_off;
    c.p0.vn = static_cast<const In *>(a.vn) + v_off;
    c.p0.g = a.g + g_off;
    c.p0.beta = a.beta + g_off;
    c.p0.gn = a.gn + g_off;
    c.p0.betan = a.betan + g_off;
    c.p0.o = static_cast<Out *>(a.o) + v_off;
    c.p0.on = static_cast<Out *>(a.on) + v_off;
    c.qks = a.h_qk * DK;
    c.vst = a.h_v * a.dv;
    c.gst = a.h_v;
    c.qk_blk = (long)a.L * c.qks;
    c.v_blk = (long)a.L * c.vst;
    c.g_blk = (long)a.L * c.gst;
    c.len = len;
    c.L = a.L;
    c.nl = a.nl;
    const long state_off = ((long)seq * a.h_v + h) * DK * a.dv + v0;
    c.h0 = a.h0 ? a.h0 + state_off : nullptr;
    if constexpr (K::kSeeds) {
        c.bs = static_cast<typename K::SeedT *>(a.bs) + (gblk0 * a.h_v + h) * DK * a.dv + v0;
        c.bs_blk = (long)a.h_v * DK * a.dv;
    } else {
        c.bs = nullptr;
        c.bs_blk = 0;
    }
    c.ht = a.ht ? a.ht + state_off : nullptr;
    c.dv = a.dv;
    c.scale = a.scale;
    K k(smem);
    k.run(c);
}

}  // namespace bdgdn
