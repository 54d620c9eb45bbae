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

#ifndef BDGDN_SCAN_LAYOUT
#define BDGDN_SCAN_LAYOUT 0x3333221100ull
#endif

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
    static constexpr int NW = 10, kThreads = 64 * NW;
    static constexpr int NB = LP / 16, DKB = DK / 16, NVB = BV / 16;
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
    // K^T for the state update is read straight from the K rows: with LDS transpose
    // loads for 16-bit operands, element by element for fp32
    static constexpr bool TR = SE == 2;
    static constexpr int V_B = al16(LP * VS * SE);
    static constexpr int TM_B = al16(LP * TS * SE);
    static constexpr int OFF_V = 4 * ROWS_B;
    static constexpr int OFF_TM = OFF_V + 2 * V_B;
    static constexpr int OFF_FAC = OFF_TM + 4 * TM_B;
    static constexpr int SET_B = OFF_FAC + 3 * 64 * 4;
    static constexpr int ST_B = al16(BV * RS * SE);
    static constexpr int DT_B = al16(BV * TS * SE);
    static constexpr int kLds = 160 * 1024;
    static constexpr bool DBUF = 2 * SET_B + 2 * ST_B + 2 * DT_B + 1024 <= kLds;
    static constexpr int NSET = DBUF ? 2 : 1;
    static constexpr int OFF_ST = NSET * SET_B;
    static constexpr int OFF_DT = OFF_ST + NSET * ST_B;
    static constexpr int OFF_DUMMY = OFF_DT + 2 * DT_B;   // sink for unassigned staging slots
    static constexpr int BYTES = OFF_DUMMY + 64 * 16;
    static_assert(BYTES <= kLds, "LDS budget");
    // Roles by wave: nibble w of kLayout (w = 0..9) is the role of wave w: 0 C, 1 N,
    // 2 O, 3 L.  Waves w, w + 4 and w + 8 share a SIMD.  The two waves of a compute role
    // take column halves 0 and 1 in wave order; L waves form the staging team in wave
    // order.
    enum { R_C = 0, R_N = 1, R_O = 2, R_L = 3 };
    static constexpr unsigned long long kLayout = BDGDN_SCAN_LAYOUT;
    static constexpr int role_of(int w) { return (int)((kLayout >> (4 * w)) & 15); }
    static constexpr int rank_of(int w)
    {
        int r = 0;
        for (int i = 0; i < w; ++i) r += role_of(i) == role_of(w);
        return r;
    }
    static constexpr int count_of(int role)
    {
        int n = 0;
        for (int i = 0; i < 10; ++i) n += role_of(i) == role;
        return n;
    }
    static_assert(count_of(R_C) == 2 && count_of(R_N) == 2 && count_of(R_O) == 2 && count_of(R_L) == 4, "layout");
    // the team of waves that loads and stages: the L waves
    static constexpr int TW = 4, TT = 64 * TW;
    static constexpr int CPR = DK / EPC;                  // chunks per q / k row
    static constexpr int OCH = LP * CPR;                  // chunks per row set
    static constexpr int OPS = (OCH + TT - 1) / TT;       // row slots per thread (x 4 sets)
    static constexpr int VCPR = BV / EPC;
    static constexpr int VPS = LP * VCPR;                 // V chunks per stream
    static_assert(VPS % 64 == 0, "a wave's V slot lies in one stream");
    static constexpr int VPL = (2 * VPS + TT - 1) / TT;   // V slots per thread (both streams)
    static constexpr int MCPR = LP / EPC, MCH = 4 * LP * MCPR;
    static constexpr int FCH = Rc::FACT_BYTES / 16;
    static constexpr int RPL = (MCH + TT - 1) / TT;       // record matrix slots per thread
    static_assert(FCH <= TT, "one factor slot");
    static_assert(Rc::OFF_EG == 16 * MCH, "factors follow the matrices");

    unsigned char *smem;
    int tid, lane, wave;

    int role, rank;   // this wave's role and its index among the waves of that role

    __device__ Scan(unsigned char *s) : smem(s)
    {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = wave_id();
        role = (int)((kLayout >> (4 * wave)) & 15);
        rank = 0;
#pragma unroll
        for (int i = 0; i < 10; ++i) rank += (i < wave && role_of(i) == role) ? 1 : 0;
    }
    __device__ __forceinline__ unsigned char *set(int p) const { return smem + p * SET_B; }
    __device__ __forceinline__ E *rows(int p, int i) const { return reinterpret_cast<E *>(set(p) + i * ROWS_B); }
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
    // The L team moves one block: 4 row sets, V and V~ (the column tile), and the
    // record.  Every thread runs the same straight-line sequence of slots (no branches,
    // so the compiler's load counters stay exact and a wait never covers loads of the
    // next block): an unassigned slot reloads the block's first chunk (a cache hit) and
    // stores it into a per-lane sink in LDS.  Resources cover exactly the block's valid
    // rows, so rows past the block end read as zero.
    struct Offs {
        unsigned rg[OPS], rl[OPS];   // row slots: global byte offset, LDS byte offset in a row set
        unsigned vg[VPL], vl[VPL];   // V slots (stream and validity are per wave)
        unsigned mg[RPL], ml[RPL];   // record matrix slots (LDS offset relative to the set)
        unsigned fg, fl;             // factor slot
    };
    // V slot u of team wave tw: stream m, or none
    __device__ __forceinline__ static int v_base(int tw, int u) { return tw * 64 + TT * u; }
    __device__ __forceinline__ void make_offs(const Chain &c, Offs &of) const
    {
        const int tw = rank, lt = 64 * tw + lane;
        const unsigned sink = (unsigned)(OFF_DUMMY + 16 * lane);
#pragma unroll
        for (int u = 0; u < OPS; ++u) {
            const int ch = lt + TT * u, t = ch / CPR, cc = ch % CPR;
            const bool ok = ch < OCH;
            of.rg[u] = ok ? (unsigned)(t * c.qks * SE + cc * 16) : 0u;
            of.rl[u] = ok ? (unsigned)((t * RS + cc * EPC) * SE) : sink;
        }
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            const int vb = v_base(tw, u);
            const bool ok = vb < 2 * VPS;
            const int ch = (ok ? vb % VPS : 0) + lane, t = ch / VCPR, cc = ch % VCPR;
            of.vg[u] = ok ? (unsigned)(t * c.vst * SE + cc * 16) : 0u;
            of.vl[u] = ok ? (unsigned)(OFF_V + (vb / VPS) * V_B + (t * VS + cc * EPC) * SE) : sink;
        }
#pragma unroll
        for (int u = 0; u < RPL; ++u) {
            const int ch = lt + TT * u;
            const bool ok = ch < MCH;
            const int m = ch / (LP * MCPR), rr = (ch / MCPR) % LP, cc = ch % MCPR;
            of.mg[u] = ok ? (unsigned)(16 * ch) : 0u;
            of.ml[u] = ok ? (unsigned)(OFF_TM + m * TM_B + (rr * TS + cc * EPC) * SE) : sink;
        }
        {
            // factor chunk e holds floats 4 e .. 4 e + 3 of [eG | dG | eGn]
            const bool ok = lt < FCH;
            const int e = 4 * lt, m = e / LP, i = e % LP;
            of.fg = ok ? (unsigned)(Rc::OFF_EG + 16 * lt) : 0u;
            of.fl = ok ? (unsigned)(OFF_FAC + (m * 64 + i) * 4) : sink;
        }
    }

    struct Fetched {
        u32x4 rb[4][OPS];
        u32x4 vb[VPL];
        u32x4 mb[RPL];
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
    __device__ __forceinline__ void st16(int p, unsigned off, u32x4 v) const
    {
        // offsets below OFF_DUMMY are inside the staging set; the sink is absolute
        unsigned char *base = off >= (unsigned)OFF_DUMMY ? smem : set(p);
        *reinterpret_cast<u32x4 *>(base + off) = v;
    }

    struct Rsrcs {
        __amdgpu_buffer_rsrc_t r[4], v[2], m;
    };
    __device__ __forceinline__ Rsrcs rsrcs(const Ptrs &P, const Chain &c, int nvalid) const
    {
        const unsigned rb = (unsigned)(nvalid * c.qks * SE), vb = (unsigned)(nvalid * c.vst * SE);
        Rsrcs r;
        r.r[0] = rsrc(P.k, rb);
        r.r[1] = rsrc(P.q, rb);
        r.r[2] = rsrc(P.kn, rb);
        r.r[3] = rsrc(P.qn, rb);
        r.v[0] = rsrc(P.v, vb);
        r.v[1] = rsrc(P.vn, vb);
        r.m = rsrc(P.rec, nvalid > 0 ? (unsigned)Rc::BYTES : 0u);
        return r;
    }

    __device__ __forceinline__ void fetch(const Ptrs &P, const Chain &c, int nvalid, const Offs &of, Fetched &f) const
    {
        const int tw = rank;
        const Rsrcs r = rsrcs(P, c, nvalid);
#pragma unroll
        for (int u = 0; u < OPS; ++u)
#pragma unroll
            for (int si = 0; si < 4; ++si) f.rb[si][u] = bload(r.r[si], of.rg[u]);
#pragma unroll
        for (int u = 0; u < VPL; ++u) f.vb[u] = bload(v_base(tw, u) >= VPS ? r.v[1] : r.v[0], of.vg[u]);
#pragma unroll
        for (int u = 0; u < RPL; ++u) f.mb[u] = bload(r.m, of.mg[u]);
        f.fb = bload(r.m, of.fg);
    }

    // Stage the fetched block into set p, refilling each register with the matching
    // chunk of the block at Pn right after it is written (nvalid_n = 0: nothing), so
    // the next block's loads are in flight while the current ones are consumed.
    __device__ __forceinline__ void stage_next(int p, Fetched &f, const Ptrs &Pn, int nvalid_n, const Chain &c,
                                               const Offs &of) const
    {
        const int tw = rank;
        const Rsrcs r = rsrcs(Pn, c, nvalid_n);
        const unsigned rset = (unsigned)ROWS_B;
#pragma unroll
        for (int u = 0; u < OPS; ++u)
#pragma unroll
            for (int si = 0; si < 4; ++si) {
                st16(p, of.rl[u] + (of.rl[u] >= (unsigned)OFF_DUMMY ? 0u : si * rset), to_operand<In, E>(f.rb[si][u]));
                f.rb[si][u] = bload(r.r[si], of.rg[u]);
            }
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            st16(p, of.vl[u], f.vb[u]);
            f.vb[u] = bload(v_base(tw, u) >= VPS ? r.v[1] : r.v[0], of.vg[u]);
        }
#pragma unroll
        for (int u = 0; u < RPL; ++u) {
            st16(p, of.ml[u], f.mb[u]);
            f.mb[u] = bload(r.m, of.mg[u]);
        }
        st16(p, of.fl, f.fb);
        f.fb = bload(r.m, of.fg);
    }

    // ------------------------------------------------------------------ helpers
    __device__ __forceinline__ f32x4 ld4f(const float *p) const { return *reinterpret_cast<const f32x4 *>(p); }

    // X = R S for the NB row tiles of row set R and NC column halves (state operand
    // quads sq[c]); each A quad is read once for all halves.
    template <int NC>
    __device__ __forceinline__ void x_rows(f32x4 (&x)[NB][NC], const E *R, const QE (&sq)[NC][DKB]) const
    {
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[DKB];
            ld_quads<E, DKB>(a, R + 16 * rb * RS, RS, lane);
#pragma unroll
            for (int c = 0; c < NC; ++c) x[rb][c] = mma_q<E, DKB>(f32x4{0.f, 0.f, 0.f, 0.f}, a, sq[c]);
        }
    }

    // D = V - diag(G) X (column halves bc0 .. bc0 + NC - 1), as B-operand quads.
    template <int NC>
    __device__ __forceinline__ void d_quads(QE (&dq)[NC][NB], const f32x4 (&x)[NB][NC], const In *V, const float *G,
                                            int bc0) const
    {
        const int g = lane >> 4, n = lane & 15;
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            const int r = 16 * rb + 4 * g;
            const f32x4 gq = ld4f(G + r);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const In *vp = V + r * VS + 16 * (bc0 + c) + n;
                f32x4 d;
#pragma unroll
                for (int i = 0; i < 4; ++i) d[i] = to_f(vp[i * VS]) - gq[i] * x[rb][c][i];
                dq[c][rb] = quad_of<E>(d);
            }
        }
    }

    // Y = M Z + init for a record matrix M (LP x LP) and B-operand quads zq[c].
    template <int NC>
    __device__ __forceinline__ void m_times(f32x4 (&y)[NB][NC], const E *M, const QE (&zq)[NC][NB],
                                            const f32x4 (&init)[NB][NC]) const
    {
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            QE a[NB];
            ld_quads<E, NB>(a, M + 16 * rb * TS, TS, lane);
#pragma unroll
            for (int c = 0; c < NC; ++c) y[rb][c] = mma_q<E, NB>(init[rb][c], a, zq[c]);
        }
    }

    // Rows at or past nvalid fall outside the store resource and are dropped.
    template <int NC>
    __device__ __forceinline__ void store_out(Out *dst, int stride, int nvalid, int bc0, const f32x4 (&acc)[NB][NC],
                                              float scale) const
    {
        constexpr int SO = (int)sizeof(Out);
        const __amdgpu_buffer_rsrc_t r = rsrc(dst, (unsigned)(nvalid * stride * SO));
        const int g = lane >> 4, n = lane & 15;
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int off = ((16 * rb + 4 * g + i) * stride + 16 * (bc0 + c) + n) * SO;
                    const Out v = to_e<Out>(acc[rb][c][i] * scale);
                    if constexpr (SO == 4)
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, 0);
                    else
                        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), r, off, 0, 0);
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
            const E *src = rows(p, 0) + 4 * (lane >> 4) * RS + 16 * kb + (lane & 15);
#pragma unroll
            for (int rb = 0; rb < NB; ++rb)
#pragma unroll
                for (int i = 0; i < 4; ++i) a[rb][i] = src[(16 * rb + i) * RS];
        }
    }

    // ------------------------------------------------------------------ roles
    // C: one block of the recurrence for column half bc.  S (fp32) and sq (its operand
    // copy) are the state on entry and on exit; Delta^T goes to dt(db).
    __device__ __forceinline__ void c_block(int p, int db, int bc, f32x4 (&S)[DKB], QE (&sq)[DKB]) const
    {
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z[NB][1] = {};
        const QE(&sq1)[1][DKB] = *reinterpret_cast<const QE(*)[1][DKB]>(&sq);
        f32x4 x[NB][1];
        x_rows<1>(x, rows(p, 0), sq1);
        QE dq[1][NB];
        d_quads<1>(dq, x, vs(p, 0), fac(p, 0), bc);
        f32x4 dl[NB][1];
        m_times<1>(dl, tm(p, 0), dq, z);
        QE uq[NB];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            st_quad(dt(db) + (16 * bc + n) * TS + 16 * rb + 4 * g, quad_of<E>(dl[rb][0]));
            uq[rb] = quad_of<E>(dl[rb][0] * ld4f(fac(p, 1) + 16 * rb + 4 * g));
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

    // N and O: one wave per column half
    static constexpr int NCP = 1;

    // N: the noisy block for column half C0 from the state operand in st(sb).
    __device__ __forceinline__ void n_block(int p, int sb, int C0, Out *on, int stride, int nvalid, float scale) const
    {
        const f32x4 z[NB][NCP] = {};
        QE sq[NCP][DKB];
#pragma unroll
        for (int c = 0; c < NCP; ++c) ld_quads<E, DKB>(sq[c], st(sb) + 16 * (C0 + c) * RS, RS, lane);
        f32x4 x3[NB][NCP], x4[NB][NCP];
        x_rows<NCP>(x3, rows(p, 2), sq);
        x_rows<NCP>(x4, rows(p, 3), sq);
        QE dq[NCP][NB];
        d_quads<NCP>(dq, x3, vs(p, 1), fac(p, 2), C0);
        f32x4 dn[NB][NCP];
        m_times<NCP>(dn, tm(p, 1), dq, z);
        QE nq[NCP][NB];
        const float gn_end = fac(p, 2)[LP - 1];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb)
#pragma unroll
            for (int c = 0; c < NCP; ++c) {
                nq[c][rb] = quad_of<E>(dn[rb][c]);
                x4[rb][c] *= gn_end;
            }
        f32x4 o[NB][NCP];
        m_times<NCP>(o, tm(p, 3), nq, x4);
        store_out<NCP>(on, stride, nvalid, C0, o, scale);
    }

    // O, first half: X2 scaled by eG for column half bc, and the P quads, kept until
    // Delta is published.
    __device__ __forceinline__ void o_begin(int p, int sb, int bc, f32x4 (&x2)[NB][1], QE (&pq)[NB][NB]) const
    {
        const int g = lane >> 4;
        QE sq[1][DKB];
        ld_quads<E, DKB>(sq[0], st(sb) + 16 * bc * RS, RS, lane);
        x_rows<1>(x2, rows(p, 1), sq);
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) {
            x2[rb][0] *= ld4f(fac(p, 0) + 16 * rb + 4 * g);
            ld_quads<E, NB>(pq[rb], tm(p, 2) + 16 * rb * TS, TS, lane);
        }
    }

    // O, second half: O = s (X2 + P Delta) with Delta^T from dt(db).
    __device__ __forceinline__ void o_end(int db, int bc, const f32x4 (&x2)[NB][1], const QE (&pq)[NB][NB], Out *o,
                                          int stride, int nvalid, float scale) const
    {
        QE dq[1][NB];
        ld_quads<E, NB>(dq[0], dt(db) + 16 * bc * TS, TS, lane);
        f32x4 acc[NB][1];
#pragma unroll
        for (int rb = 0; rb < NB; ++rb) acc[rb][0] = mma_q<E, NB>(x2[rb][0], pq[rb], dq[0]);
        store_out<1>(o, stride, nvalid, bc, acc, scale);
    }

    // ------------------------------------------------------------------ the chain
    // Waves by the layout table: C, N, O (column half = rank), L.  With one
    // staging set, L stages each block in a phase of its own (the other waves wait at
    // a barrier) and C publishes the state operand in that phase.
    __device__ void run(const Chain &c) const
    {
        const int nb = (int)((c.len + c.L - 1) / c.L);
        const int g = lane >> 4, n = lane & 15;
        if (role == R_C) {
            // ---- C
            const int bc = rank;
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
            if (DBUF) write_st(0, sq, bc);
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                if (!DBUF) {
                    write_st(0, sq, bc);
                    lds_barrier();
                }
                c_block(DBUF ? (j & 1) : 0, j & 1, bc, S, sq);
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
        } else if (role == R_N) {
            // ---- N
            const int bc = rank;
            Ptrs pc = c.p0;
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                if (!DBUF) lds_barrier();
                n_block(DBUF ? (j & 1) : 0, DBUF ? (j & 1) : 0, bc, pc.on, c.vst, nvalid_of(c, j), c.scale);
                advance(pc, c);
                lds_barrier();
            }
        } else if (role == R_O) {
            // ---- O
            const int bc = rank;
            Ptrs pc = c.p0;
            f32x4 x2[NB][1];
            QE pq[NB][NB];
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                if (!DBUF) lds_barrier();
                if (j > 0) {
                    o_end((j - 1) & 1, bc, x2, pq, pc.o, c.vst, nvalid_of(c, j - 1), c.scale);
                    advance(pc, c);
                }
                o_begin(DBUF ? (j & 1) : 0, DBUF ? (j & 1) : 0, bc, x2, pq);
                lds_barrier();
            }
            if (nb > 0) o_end((nb - 1) & 1, bc, x2, pq, pc.o, c.vst, nvalid_of(c, nb - 1), c.scale);
        } else {
            // ---- L
            Offs of;
            make_offs(c, of);
            Ptrs pf = c.p0;   // next block to load
            auto nv = [&](int jj) { return jj < nb ? nvalid_of(c, jj) : 0; };
            if constexpr (DBUF && SE == 4) {
                // fp32: step j stages block j + 1 and loads block j + 2
                Fetched f;
                fetch(pf, c, nv(0), of, f);
                advance(pf, c);
                if (nb > 0) stage_next(0, f, pf, nv(1), c, of);
                advance(pf, c);
                lds_barrier();
                for (int j = 0; j < nb; ++j) {
                    if (j + 1 < nb) stage_next((j + 1) & 1, f, pf, nv(j + 2), c, of);
                    advance(pf, c);
                    lds_barrier();
                }
            } else if constexpr (DBUF) {
                // step j stages block j + 1 from f[(j + 1) & 1] and loads block j + 3 into it:
                // two blocks of loads in flight
                Fetched f0, f1;
                fetch(pf, c, nv(0), of, f0);
                advance(pf, c);
                fetch(pf, c, nv(1), of, f1);
                advance(pf, c);
                if (nb > 0) stage_next(0, f0, pf, nv(2), c, of);   // block 0; f0 <- block 2
                advance(pf, c);
                lds_barrier();
                for (int j = 0; j < nb; j += 2) {
                    if (j + 1 < nb) stage_next(1, f1, pf, nv(j + 3), c, of);
                    advance(pf, c);
                    lds_barrier();
                    if (j + 1 < nb) {
                        if (j + 2 < nb) stage_next(0, f0, pf, nv(j + 4), c, of);
                        advance(pf, c);
                        lds_barrier();
                    }
                }
            } else {
                // one set: step j stages block j in a phase of its own, loading block j + 1
                Fetched f;
                fetch(pf, c, nv(0), of, f);
                advance(pf, c);
                lds_barrier();
                for (int j = 0; j < nb; ++j) {
                    stage_next(0, f, pf, nv(j + 1), c, of);
                    advance(pf, c);
                    lds_barrier();
                    lds_barrier();
                }
            }
        }
    }
};

}  // namespace bdgdn
