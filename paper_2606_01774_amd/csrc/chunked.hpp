// chunked.hpp -- the chunk-parallel two-stream training forward (Appendix "Route II",
// alg. route-twostream-fwd with the chunk-state pass of eq. chunk-state): the sequence of
// every (sequence or document, v-head) chain is cut into segments of G blocks, the clean
// state at each segment start is found first by a light serial pass, and then every
// (chain, segment) is evaluated in parallel, all d_v columns in one workgroup.
//
// Three kernels:
//   rec     per (block, v-head) of the state pass, in parallel: the clean block-local UT
//           transform T = (I + A)^(-1) diag(beta) and the gate factors eG = gamma_r,
//           dG = gamma_n / gamma_r (Appendix "Chunk-corrected values", eq. f-blk);
//   states  per (chain, 32-column tile of d_v): the clean recurrence in block form,
//             Delta = T (V - diag(eG) K S0),  S <- gamma_n S0 + K^T diag(dG) Delta,
//           over the blocks before the last segment, writing S at every segment start
//           (the chunk-state pass, eq. chunk-state); no outputs;
//   out     per (chain, segment): from the segment's start state, every block's clean
//           outputs O = diag(eG) Q S0 + P Delta, its noisy outputs
//           O~ = gamma~_n Q~ S0 + R Delta~ (eq. noisy-block-fwd, the noisy block seeded
//           with the clean state at its start) and the clean state update, with
//             P_rc = 2^(G_r - G_c) (q_r . k_c) (c <= r),  R_rc = 2^(G~_n - G~_c) (q~_r . k~_c).
//
// The out kernel gives each of its C waves 16 columns of the state, held in registers
// (fp32, with its fp16 operand copy), and that wave forms every product with the state for
// its columns: no state goes through LDS, and everything independent of d_v (the rows of
// the block converted to fp16, T, T~, P, R) is staged or computed once per block for all
// columns.  Per block j of the segment, with one workgroup barrier per block:
//   C (NC waves)  block j: its 16 columns of O, O~ and of the state update
//   U0, U1        the clean (T, P, factors) and noisy (T~, R, factors) records of block j + 1
//   L (NL waves)  the rows of block j + 2 into a three-slot ring, V and V~ of block j + 1
#pragma once

#include "intra.hpp"
#include "kernels.hpp"
#include "ut.hpp"

namespace bdgdn {

namespace chunked {

typedef __bf16 In;
typedef _Float16 E;
typedef Quad<E> QE;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, unsigned bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 bload(__amdgpu_buffer_rsrc_t r, unsigned off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}
__device__ __forceinline__ f32x4 ld4f(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }

// Byte layout of one clean record of the state pass: T and N = K_(j+1) K_j^T (fp16, LP x LP
// row-major each; N is zero for the chain's last scanned block), eG, dG (fp32, LP each).
template <int LP> struct CRec {
    static constexpr int OFF_T = 0, OFF_N = LP * LP * 2, OFF_EG = 2 * LP * LP * 2, OFF_DG = OFF_EG + LP * 4;
    static constexpr int BYTES = al256(OFF_DG + LP * 4);
};

// Geometry of the segments, shared by the three kernels.
struct Geo {
    long base, len;   // first row and rows of the chain's sequence or document
    int nb;           // blocks of the chain
    int nseg;         // segments of G blocks
    int doc;          // sequence / document index
    int pos;          // its position in the processing order
};
// An empty document is one segment without blocks (its unit writes ht = h0).
__device__ __forceinline__ int nseg_of(int nb, int G) { return nb <= 0 ? 1 : (nb + G - 1) / G; }
__device__ __forceinline__ Geo geo_of(const ChunkArgs &a, int pos)
{
    Geo r;
    r.pos = pos;
    if (a.cu) {
        r.doc = a.n_order > 0 ? (a.order[pos] & 1023) : pos;
        r.base = a.cu[r.doc];
        r.len = (long)a.cu[r.doc + 1] - r.base;
    } else {
        r.doc = pos;
        r.base = (long)pos * a.T;
        r.len = a.T;
    }
    r.nb = (int)((r.len + a.L - 1) / a.L);
    r.nseg = nseg_of(r.nb, a.G);
    return r;
}
// Segments of the documents before position pos in the processing order.
__device__ __forceinline__ int segs_before(const ChunkArgs &a, int pos)
{
    return a.cu ? (int)((unsigned)a.order[pos] >> 10) : pos * nseg_of(a.nblk, a.G);
}
// Dense indices of the state pass's records and checkpoints: the chains of the first n1
// positions in order, position by position, each v-head of a position holding (nseg - 1)
// checkpoints and (nseg - 1) G records.  Every position before pos has two or more
// segments, so the checkpoints before it number segs_before(pos) - pos per v-head.
__device__ __forceinline__ long ckpt_base(const ChunkArgs &a, int pos, int h, int nseg)
{
    return (long)(segs_before(a, pos) - pos) * a.h_v + (long)h * (nseg - 1);
}
__device__ __forceinline__ long ckpt_index(const ChunkArgs &a, int pos, int h, int nseg, int s)
{
    return ckpt_base(a, pos, h, nseg) + (s - 1);
}
__device__ __forceinline__ long rec_index(const ChunkArgs &a, int pos, int h, int nseg, int j)
{
    return ckpt_base(a, pos, h, nseg) * a.G + j;
}

// Workgroup ids are dealt to the GPU's eight XCDs in turn, each with its own L2.  The state
// pass's chains are padded to a multiple of 8 and laid out so that every workgroup of chain
// c (its record groups, its d_v tiles) has an id congruent to c mod 8: a chain's key rows
// and records are read through one L2.
__device__ __forceinline__ int chains_padded(const ChunkArgs &a) { return (a.n1 * a.h_v + 7) & ~7; }

// Element offset of (row, k) in a swizzled [rows][DK] fp16 matrix: chunk k/8 of a row is
// stored at chunk (k/8) ^ (row / RPB mod CPR).
template <int DK> struct Swz {
    static constexpr int CPR = DK / 8, RPB = 256 / (2 * DK);
    __device__ __forceinline__ static int rofs(int row, int k)
    {
        return row * DK + ((((k >> 3) ^ ((row / RPB) & (CPR - 1))) << 3) | (k & 7));
    }
};

// Per-lane offsets of the operand quads of a 16-row block (row lane & 15, k-block kb) and
// of the transpose-load segments of K^T.
template <int DK> struct QOffs {
    static constexpr int DKB = DK / 16;
    int q[DKB], t[DKB];
    __device__ __forceinline__ void make(int lane)
    {
        const int r = lane & 15, g = lane >> 4;
        const int tr = 4 * g + ((lane >> 2) & 3), tq = lane & 3;
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) {
            q[kb] = Swz<DK>::rofs(r, 16 * kb + 4 * g);
            t[kb] = Swz<DK>::rofs(tr, 16 * kb + 4 * tq);
        }
    }
};
template <int NKB, int DK>
__device__ __forceinline__ void ld_q(QE (&q)[NKB], const E *M, const int (&off)[DK / 16])
{
    typedef const __attribute__((address_space(3))) volatile QE *LQ;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) q[kb] = *(LQ)(M + off[kb]);
}
// A-operand quads of K^T rows 16 kb .. 16 kb + 15 from swizzled K rows (transpose loads).
template <int NB, int DK>
__device__ __forceinline__ void kt_quads(QE (&a)[NB], const E *K, int kb, const QOffs<DK> &qo)
{
#pragma unroll
    for (int rb = 0; rb < NB; ++rb)
        a[rb] = __builtin_bit_cast(QE, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                           (__attribute__((address_space(3))) s16x4 *)(K + 16 * rb * DK + qo.t[kb])));
}

// Store an output tile pair (rows 16 rb + 4g + i, column c0 + n) scaled.
template <typename Out, int NB>
__device__ __forceinline__ void store_out(Out *dst, int stride, int nvalid, int c0, const f32x4 (&acc)[NB], float scale,
                                          int lane)
{
    constexpr int SO = (int)sizeof(Out);
    const __amdgpu_buffer_rsrc_t r = rsrc(dst, (unsigned)(nvalid * stride * SO));
    const int g = lane >> 4, n = lane & 15;
#pragma unroll
    for (int rb = 0; rb < NB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int off = ((16 * rb + 4 * g + i) * stride + c0 + n) * SO;
            const Out v = to_e<Out>(acc[rb][i] * scale);
            if constexpr (SO == 4)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, off, 0, 0);
            else
                __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), r, off, 0, 0);
        }
}

// ====================================================================== rec
// One workgroup per (state-pass chain, group of four blocks): the key rows of the four
// blocks and of the block after them are staged once (fp16, swizzled), then wave w writes
// the record of block j0 + w: its gate factors, T and N = K_(j+1) K_j^T.
template <int DK, int LP>
struct RecKernel {
    static constexpr int NB = LP / 16, DKB = DK / 16;
    typedef CRec<LP> R;
    typedef Swz<DK> SW;
    static constexpr int kWaves = 4, kThreads = 64 * kWaves;
    static constexpr int NR = (kWaves + 1) * LP;             // staged rows
    static constexpr int ROWS_B = NR * DK * 2;
    static constexpr int OFF_G = ROWS_B;                      // per wave: cumulative gates, beta
    static constexpr int BYTES = OFF_G + kWaves * 2 * 64 * 4;
    static constexpr int CH = NR * DK / 8;                    // 16-byte chunks of the rows
    static constexpr int PER = (CH + kThreads - 1) / kThreads;

    __device__ static void run(const ChunkArgs &a, unsigned char *smem)
    {
        const int lane = threadIdx.x & 63, wave = wave_id(), tid = threadIdx.x;
        const int np = chains_padded(a);
        const int c = blockIdx.x % np, j0 = (blockIdx.x / np) * kWaves;
        if (c >= a.n1 * a.h_v) return;
        const int pos = c / a.h_v, h = c % a.h_v;
        const Geo geo = geo_of(a, pos);
        const int J = (geo.nseg - 1) * a.G;   // blocks scanned by the state pass (all full)
        if (j0 >= J) return;
        const int hq = h / (a.h_v / a.h_qk);
        const int qks = a.h_qk * DK;
        // rows j0 L .. (j0 + 5) L - 1 of the chain, those of blocks < J only
        const int nrows = (J - j0 >= kWaves + 1 ? kWaves + 1 : J - j0) * a.L;
        const In *kp = static_cast<const In *>(a.k) + ((geo.base + (long)j0 * a.L) * a.h_qk + hq) * DK;
        const __amdgpu_buffer_rsrc_t rk = rsrc(kp, (unsigned)(nrows * qks * 2));
        E *Ks = reinterpret_cast<E *>(smem);
        u32x4 f[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int ch = tid + kThreads * u, t = ch / (DK / 8), cc = ch % (DK / 8);
            // rows of the LP-padded blocks: row t of the staging is position t % LP of block t / LP
            const int gr = (t / LP) * a.L + (t % LP);
            const bool ok = ch < CH && (t % LP) < a.L;
            f[u] = bload(rk, ok ? (unsigned)(gr * qks * 2 + cc * 16) : 0x80000000u);
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int ch = tid + kThreads * u, t = ch / (DK / 8), cc = ch % (DK / 8);
            if (ch < CH) *reinterpret_cast<u32x4 *>(Ks + SW::rofs(t, 8 * cc)) = to_operand<In, E>(f[u]);
        }
        __syncthreads();
        const int j = j0 + wave;
        if (j >= J) return;
        float *Gs = reinterpret_cast<float *>(smem + OFF_G) + wave * 128, *Bs = Gs + 64;
        unsigned char *rec = a.rec + rec_index(a, pos, h, geo.nseg, j) * R::BYTES;
        const long r0 = geo.base + (long)j * a.L;
        float gv = 0.f, bv = 0.f;
        if (lane < a.L) {
            gv = a.g[(r0 + lane) * a.h_v + h];
            bv = a.beta[(r0 + lane) * a.h_v + h];
        }
        const float x = ut::scan32(lane < LP ? gv * kLog2e : 0.f, lane);
        const float gl = ut::lane_value(x, LP - 1);
        Gs[lane] = x;
        Bs[lane] = bv;
        if (lane < LP) {
            reinterpret_cast<float *>(rec + R::OFF_EG)[lane] = fexp2(x);
            reinterpret_cast<float *>(rec + R::OFF_DG)[lane] = fexp2(gl - x);
        }
        QOffs<DK> qo;
        qo.make(lane);
        const E *K = Ks + wave * LP * DK;
        ut::Consts us;
        ut::make_consts(us, lane);
        {
            QE kq[NB][DKB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) ld_q<DKB, DK>(kq[rb], K + 16 * rb * DK, qo.q);
            ut::solve_t<NB, DKB>(kq, Gs, Bs, reinterpret_cast<E *>(rec + R::OFF_T), LP, us, lane);
        }
        // N = K_(j+1) K_j^T from the transposed tiles K_j K_(j+1)^T: lane (g, n) holds entry
        // (16 br + n, 16 bc + 4g + i), four consecutive entries of one row
        E *N = reinterpret_cast<E *>(rec + R::OFF_N);
        const int g = lane >> 4, n = lane & 15;
        const bool last = j + 1 >= J;
#pragma unroll
        for (int br = 0; br < NB; ++br) {
            QE kn[DKB];
            ld_q<DKB, DK>(kn, K + (LP + 16 * br) * DK, qo.q);
#pragma unroll
            for (int bc = 0; bc < NB; ++bc) {
                QE kc[DKB];
                ld_q<DKB, DK>(kc, K + 16 * bc * DK, qo.q);
                f32x4 v = mma_q<E, DKB>(f32x4{0.f, 0.f, 0.f, 0.f}, kc, kn);
                if (last) v = f32x4{0.f, 0.f, 0.f, 0.f};
                st_quad(N + (16 * br + n) * LP + 16 * bc + 4 * g, quad_of<E>(v));
            }
        }
    }
};

// ====================================================================== states
// One workgroup per (state-pass chain, 32-column tile): waves 0, 1 scan 16 columns each,
// waves 2, 3 stage every block's key rows (fp16), V tile and record three blocks ahead
// into a four-slot ring.
//
// The scan carries X_j = K_j S_j, the keys times the state at the block start, and uses
//     X_(j+1) = K_(j+1) S_(j+1) = gamma_n K_(j+1) S_j + (K_(j+1) K_j^T) diag(dG) Delta_j,
// so that per block only Delta_j = T (V - diag(eG) X_j) and the short product with N_j stand
// between one block and the next; the state update S_(j+1) = gamma_n S_j + K_j^T diag(dG)
// Delta_j and Y_(j+2) = K_(j+2) S_(j+1) are off that path.
template <int DK, int LP>
struct StatesKernel {
    static constexpr int NB = LP / 16, DKB = DK / 16, BV = 32;
    static constexpr int kThreads = 256;
    typedef Swz<DK> SW;
    typedef CRec<LP> R;
    static constexpr int TS = LP + 8, VS = BV + 8;
    static constexpr int ROWS_B = LP * DK * 2;
    static constexpr int V_B = al16(LP * VS * 2);
    static constexpr int M_B = al16(LP * TS * 2);
    static constexpr int OFF_V = ROWS_B, OFF_T = OFF_V + V_B, OFF_N = OFF_T + M_B, OFF_F = OFF_N + M_B;
    static constexpr int SLOT_B = al16(OFF_F + 2 * LP * 4);
    static constexpr int NS = 4;                   // LDS slots: blocks j .. j + 2 in use, j + 3 staged
    static constexpr int OFF_SINK = NS * SLOT_B;
    static constexpr int BYTES = OFF_SINK + 16 * 128;
    // staging: chunks of 16 bytes per block
    static constexpr int TT = 128;
    static constexpr int KCH = LP * DK / 8;        // key rows
    static constexpr int VCH = LP * BV / 8;        // V tile
    static constexpr int MCH = LP * LP / 8;        // T or N
    static constexpr int FCH = 2 * LP / 4;         // eG, dG
    static constexpr int NCH = KCH + VCH + 2 * MCH + FCH;
    static constexpr int PER = (NCH + TT - 1) / TT;
    static constexpr int NREG = 3;                 // blocks of loads in flight per L lane
    static_assert(KCH % 64 == 0 && VCH % 64 == 0, "wave-uniform staging sources");

    struct Slots {
        unsigned g[PER];          // byte offset in its source (rows, V, or the record)
        unsigned l[PER];          // LDS byte offset in a slot (or the sink)
        unsigned char src[PER];   // 0 rows, 1 V, 2 record
    };
    struct Regs {
        u32x4 c[PER];
    };

    __device__ static void run(const ChunkArgs &a, unsigned char *smem)
    {
        const int lane = threadIdx.x & 63, wave = wave_id();
        const int per = 8 * a.n_vt, rem = blockIdx.x % per;
        const int c = (blockIdx.x / per) * 8 + rem % 8, vt = rem / 8;
        if (c >= a.n1 * a.h_v) return;
        const int pos = c / a.h_v, h = c % a.h_v;
        const Geo geo = geo_of(a, pos);
        const int J = (geo.nseg - 1) * a.G;   // blocks scanned
        if (J <= 0) return;
        const int hq = h / (a.h_v / a.h_qk);
        const int v0 = vt * BV;
        const In *kp = static_cast<const In *>(a.k) + (geo.base * a.h_qk + hq) * DK;
        const In *vp = static_cast<const In *>(a.v) + (geo.base * a.h_v + h) * a.dv + v0;
        const unsigned char *recp = a.rec + rec_index(a, pos, h, geo.nseg, 0) * R::BYTES;
        const int qks = a.h_qk * DK, vst = a.h_v * a.dv;
        if (wave < 2) {
            // ---- C: 16 columns
            const int g = lane >> 4, n = lane & 15;
            const int c0 = v0 + 16 * wave;
            QOffs<DK> qo;
            qo.make(lane);
            f32x4 S[DKB];
            QE sq[DKB];
            const float *h0 = a.h0 ? a.h0 + ((long)geo.doc * a.h_v + h) * DK * a.dv + c0 : nullptr;
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                f32x4 s = {0.f, 0.f, 0.f, 0.f};
                if (h0) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) s[i] = h0[(long)(16 * kb + 4 * g + i) * a.dv + n];
                }
                S[kb] = s;
                sq[kb] = quad_of<E>(s);
            }
            lds_barrier();
            lds_barrier();
            const f32x4 z = {0.f, 0.f, 0.f, 0.f};
            auto slot_of = [&](int jj) { return smem + (jj % NS) * SLOT_B; };
            auto krows = [&](f32x4 (&y)[NB], int jj) {   // y = K_jj S (state operand sq)
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) {
                    QE kq[DKB];
                    ld_q<DKB, DK>(kq, reinterpret_cast<const E *>(slot_of(jj)) + 16 * rb * DK, qo.q);
                    y[rb] = mma_q<E, DKB>(z, kq, sq);
                }
            };
            // the operands of the serial path of block jj, read from LDS a step ahead
            struct Ops {
                f32x4 v[NB];           // V tile, this wave's column
                f32x4 eg[NB], dg[NB];  // gate factors of rows 16 rb + 4g + i
                QE t[NB][NB], nm[NB][NB];
                float decay;
            };
            auto load_ops = [&](Ops &op, int jj) {
                const unsigned char *sl = slot_of(jj);
                const In *V = reinterpret_cast<const In *>(sl + OFF_V);
                const float *eG = reinterpret_cast<const float *>(sl + OFF_F), *dG = eG + LP;
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) {
                    const int rr = 16 * rb + 4 * g;
#pragma unroll
                    for (int i = 0; i < 4; ++i) op.v[rb][i] = to_f(V[(rr + i) * VS + 16 * wave + n]);
                    op.eg[rb] = ld4f(eG + rr);
                    op.dg[rb] = ld4f(dG + rr);
                    ld_quads<E, NB>(op.t[rb], reinterpret_cast<const E *>(sl + OFF_T) + 16 * rb * TS, TS, lane);
                    ld_quads<E, NB>(op.nm[rb], reinterpret_cast<const E *>(sl + OFF_N) + 16 * rb * TS, TS, lane);
                }
                op.decay = eG[LP - 1];
            };
            f32x4 x[NB], y[NB];
            krows(x, 0);   // X_0 = K_0 S_0
            krows(y, 1);   // Y_1 = K_1 S_0
            Ops op;
            load_ops(op, 0);
            int s_next = a.G;
            for (int j = 0; j < J; ++j) {
                const E *K = reinterpret_cast<const E *>(slot_of(j));
                // serial path: Delta_j = T (V - diag(eG) X_j), uq = diag(dG) Delta_j,
                // X_(j+1) = gamma_n Y_(j+1) + N_j uq
                QE dq[NB];
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) dq[rb] = quad_of<E>(op.v[rb] - op.eg[rb] * x[rb]);
                QE uq[NB];
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) uq[rb] = quad_of<E>(mma_q<E, NB>(z, op.t[rb], dq) * op.dg[rb]);
                const float decay = op.decay;
#pragma unroll
                for (int rb = 0; rb < NB; ++rb) x[rb] = mma_q<E, NB>(y[rb] * decay, op.nm[rb], uq);
                load_ops(op, j + 1);
                // S_(j+1) = gamma_n S_j + K_j^T diag(dG) Delta_j
#pragma unroll
                for (int kb = 0; kb < DKB; ++kb) {
                    QE kt[NB];
                    kt_quads<NB, DK>(kt, K, kb, qo);
                    S[kb] = mma_q<E, NB>(S[kb] * decay, kt, uq);
                    sq[kb] = quad_of<E>(S[kb]);
                }
                // Y_(j+2) = K_(j+2) S_(j+1)
                krows(y, j + 2);
                if (j + 1 == s_next) {
                    write_ckpt(a, pos, h, geo.nseg, s_next / a.G, c0, S, lane);
                    s_next += a.G;
                }
                lds_barrier();
            }
        } else {
            // ---- L: step j stores the loads of block j + 3 and loads block j + 3 + NREG
            const int lt = 64 * (wave - 2) + lane;
            Slots sl;
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                int ch = lt + TT * u;
                unsigned gsrc = 0, lds = (unsigned)(OFF_SINK + 16 * lt);
                int src = 2;   // past the chunks: reload the record's first chunk into the sink
                if (ch < KCH) {
                    const int t = ch / (DK / 8), cc = ch % (DK / 8);
                    gsrc = (unsigned)(t * qks * 2 + cc * 16);
                    lds = (unsigned)(2 * SW::rofs(t, 8 * cc));
                    src = 0;
                } else if ((ch -= KCH) < VCH) {
                    const int t = ch / (BV / 8), cc = ch % (BV / 8);
                    gsrc = (unsigned)(t * vst * 2 + cc * 16);
                    lds = (unsigned)(OFF_V + (t * VS + 8 * cc) * 2);
                    src = 1;
                } else if ((ch -= VCH) < 2 * MCH) {
                    const int m = ch / MCH, cm = ch % MCH, t = cm / (LP / 8), cc = cm % (LP / 8);
                    gsrc = (unsigned)((m ? R::OFF_N : R::OFF_T) + (t * LP + 8 * cc) * 2);
                    lds = (unsigned)((m ? OFF_N : OFF_T) + (t * TS + 8 * cc) * 2);
                } else if ((ch -= 2 * MCH) < FCH) {
                    gsrc = (unsigned)(R::OFF_EG + 16 * ch);
                    lds = (unsigned)(OFF_F + 16 * ch);
                }
                sl.g[u] = gsrc;
                sl.l[u] = lds;
                // every source boundary (KCH, KCH + VCH) is a multiple of 64 chunks, so a
                // wave's slot u reads one source
                sl.src[u] = (unsigned char)__builtin_amdgcn_readfirstlane(src);
            }
            auto fetch = [&](int jj, Regs &rg) {
                // blocks past J (never stored into a slot that is read) load block 0 again
                const int jc = jj < J ? jj : 0;
                const unsigned rb = (unsigned)(a.L * qks * 2), vb = (unsigned)(a.L * vst * 2);
                const __amdgpu_buffer_rsrc_t rr = rsrc(kp + (long)jc * a.L * qks, rb);
                const __amdgpu_buffer_rsrc_t rv = rsrc(vp + (long)jc * a.L * vst, vb);
                const __amdgpu_buffer_rsrc_t rc = rsrc(recp + (long)jc * R::BYTES, R::BYTES);
#pragma unroll
                for (int u = 0; u < PER; ++u)
                    rg.c[u] = bload(sl.src[u] == 0 ? rr : sl.src[u] == 1 ? rv : rc, sl.g[u]);
            };
            auto store = [&](int jj, Regs &rg) {
                unsigned char *base = smem + (jj % NS) * SLOT_B;
#pragma unroll
                for (int u = 0; u < PER; ++u) {
                    unsigned char *b = sl.l[u] >= (unsigned)OFF_SINK ? smem : base;
                    if (sl.src[u] == 0)
                        *reinterpret_cast<u32x4 *>(b + sl.l[u]) = to_operand<In, E>(rg.c[u]);
                    else
                        *reinterpret_cast<u32x4 *>(b + sl.l[u]) = rg.c[u];
                }
            };
            Regs r[NREG];
#pragma unroll
            for (int i = 0; i < NREG; ++i) fetch(i, r[i]);
            // blocks 0, 1 and 2 before the loop
            store(0, r[0]);
            fetch(NREG, r[0]);
            store(1, r[1]);
            fetch(NREG + 1, r[1]);
            store(2, r[2]);
            fetch(NREG + 2, r[2]);
            lds_barrier();
            lds_barrier();
            // step j stores block j + 3 (held in r[j % NREG]) and refills it with block j + 3 + NREG
            int j = 0;
            for (; j + NREG <= J; j += NREG) {
#pragma unroll
                for (int u = 0; u < NREG; ++u) {
                    store(j + u + 3, r[u]);
                    fetch(j + u + 3 + NREG, r[u]);
                    lds_barrier();
                }
            }
            for (; j < J; ++j) lds_barrier();
        }
    }
    __device__ __forceinline__ static void write_ckpt(const ChunkArgs &a, int pos, int h, int nseg, int s, int c0,
                                                      const f32x4 (&S)[DKB], int lane)
    {
        const int g = lane >> 4, n = lane & 15;
        float *dst = a.ckpt + ckpt_index(a, pos, h, nseg, s) * DK * a.dv + c0 + n;
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) dst[(long)(16 * kb + 4 * g + i) * a.dv] = S[kb][i];
    }
};

// ====================================================================== out
// One workgroup per (chain, segment, tile of DV columns of d_v).  Waves: 0 .. NC-1 C (16
// columns each), NC U0 (clean record), NC + 1 U1 (noisy record), then NL staging waves.
template <typename Out, int DK, int DV_, int LP, int NL>
struct OutKernel {
    static constexpr int DV = DV_, DK_ = DK;   // DV: the d_v columns of one workgroup
    typedef Out OutT;
    static constexpr int NB = LP / 16, DKB = DK / 16, NC = DV / 16;
    static constexpr int NW = NC + 2 + NL, kThreads = 64 * NW;
    typedef Swz<DK> SW;
    static constexpr int TS = LP + 8, VS = DV + 8;
    static constexpr int ROWS_B = LP * DK * 2;          // one row set (k, q, k~ or q~)
    static constexpr int RING_B = 4 * ROWS_B;           // one ring slot
    static constexpr int V_B = al16(LP * VS * 2);       // V or V~, bf16 [LP][VS]
    static constexpr int VSET_B = 2 * V_B;
    static constexpr int M_B = al16(LP * TS * 2);       // T, T~, P, R, fp16 [LP][TS]
    static constexpr int NFAC = 5;                      // eG, dG, G, eG~, dG~
    static constexpr int REC_B = 4 * M_B + NFAC * 64 * 4;
    static constexpr int OFF_VS = 3 * RING_B;
    static constexpr int OFF_REC = OFF_VS + 2 * VSET_B;
    static constexpr int OFF_US = OFF_REC + 2 * REC_B;
    static constexpr int OFF_SINK = OFF_US + 2 * 2 * 64 * 4;
    static constexpr int BYTES = OFF_SINK + 16 * 64 * NL;
    static_assert(BYTES <= 160 * 1024, "LDS budget");
    // staging
    static constexpr int TT = 64 * NL;
    static constexpr int OCH = LP * DK / 8;             // chunks per row set
    static constexpr int OPS = (OCH + TT - 1) / TT;
    static constexpr int VCH = LP * DV / 8;             // chunks per V stream
    static constexpr int VPL = (2 * VCH + TT - 1) / TT;
    static_assert(VCH % 64 == 0, "a wave's V slot lies in one stream");

    unsigned char *smem;
    int lane, wave;

    __device__ OutKernel(unsigned char *s) : smem(s)
    {
        lane = threadIdx.x & 63;
        wave = wave_id();
    }
    __device__ __forceinline__ E *rows(int slot, int i) const
    {
        return reinterpret_cast<E *>(smem + slot * RING_B + i * ROWS_B);
    }
    __device__ __forceinline__ In *vs(int p, int m) const
    {
        return reinterpret_cast<In *>(smem + OFF_VS + p * VSET_B + m * V_B);
    }
    __device__ __forceinline__ E *mat(int p, int m) const   // 0 T, 1 T~, 2 P, 3 R
    {
        return reinterpret_cast<E *>(smem + OFF_REC + p * REC_B + m * M_B);
    }
    __device__ __forceinline__ float *fac(int p, int m) const   // 0 eG, 1 dG, 2 G, 3 eG~, 4 dG~
    {
        return reinterpret_cast<float *>(smem + OFF_REC + p * REC_B + 4 * M_B) + 64 * m;
    }
    __device__ __forceinline__ float *us(int u) const { return reinterpret_cast<float *>(smem + OFF_US) + 128 * u; }

    struct Ptrs {
        const In *k, *q, *kn, *qn, *v, *vn;
        const float *g, *beta, *gn, *betan;
        Out *o, *on;
    };
    struct Seg {
        Ptrs p0;              // at the segment's first block
        long qk_blk, v_blk, g_blk;
        int qks, vst, gst;
        long len;             // rows from the segment start to the chain's end
        int nb;               // blocks of the segment
        int L;
        const float *s0;      // start state (column 0), or null (zero)
        float *ht;            // final state, or null
        int dv;
        float scale;
    };
    __device__ __forceinline__ static void advance(Ptrs &p, const Seg &c)
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
    __device__ __forceinline__ static int nvalid_of(const Seg &c, int j)
    {
        if (j >= c.nb) return 0;
        const long rem = c.len - (long)j * c.L;
        return rem <= 0 ? 0 : rem < c.L ? (int)rem : c.L;
    }

    // ------------------------------------------------------------------ L: staging
    struct LOffs {
        unsigned rg[OPS], rl[OPS];
        unsigned vg[VPL], vl[VPL];
        unsigned char vm[VPL];
    };
    struct RowsF {
        u32x4 c[4][OPS];
    };
    struct VF {
        u32x4 c[VPL];
    };
    __device__ __forceinline__ void make_loffs(const Seg &c, int tw, LOffs &o) const
    {
        const int lt = 64 * tw + lane;
        const unsigned sink = (unsigned)(OFF_SINK + 16 * lt);
#pragma unroll
        for (int u = 0; u < OPS; ++u) {
            const int ch = lt + TT * u, t = ch / (DK / 8), cc = ch % (DK / 8);
            const bool ok = ch < OCH;
            o.rg[u] = ok ? (unsigned)(t * c.qks * 2 + cc * 16) : 0u;
            o.rl[u] = ok ? (unsigned)(2 * SW::rofs(t, 8 * cc)) : sink;
        }
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            const int ch = lt + TT * u;
            const bool ok = ch < 2 * VCH;
            const int m = ok ? ch / VCH : 0, cv = ok ? ch % VCH : 0, t = cv / (DV / 8), cc = cv % (DV / 8);
            o.vg[u] = (unsigned)(t * c.vst * 2 + cc * 16);
            o.vl[u] = ok ? (unsigned)(m * V_B + (t * VS + 8 * cc) * 2) : sink;
            o.vm[u] = (unsigned char)__builtin_amdgcn_readfirstlane(m);   // VCH is a multiple of 64
        }
    }
    __device__ __forceinline__ void fetch_rows(const Ptrs &P, const Seg &c, int nvalid, const LOffs &o, RowsF &f) const
    {
        const unsigned b = (unsigned)(nvalid * c.qks * 2);
        const __amdgpu_buffer_rsrc_t r[4] = {rsrc(P.k, b), rsrc(P.q, b), rsrc(P.kn, b), rsrc(P.qn, b)};
#pragma unroll
        for (int u = 0; u < OPS; ++u)
#pragma unroll
            for (int si = 0; si < 4; ++si) f.c[si][u] = bload(r[si], o.rg[u]);
    }
    __device__ __forceinline__ void fetch_v(const Ptrs &P, const Seg &c, int nvalid, const LOffs &o, VF &f) const
    {
        const unsigned b = (unsigned)(nvalid * c.vst * 2);
        const __amdgpu_buffer_rsrc_t r0 = rsrc(P.v, b), r1 = rsrc(P.vn, b);
#pragma unroll
        for (int u = 0; u < VPL; ++u) f.c[u] = bload(o.vm[u] ? r1 : r0, o.vg[u]);
    }
    __device__ __forceinline__ void st16(unsigned char *base, unsigned off, u32x4 v) const
    {
        unsigned char *b = off >= (unsigned)OFF_SINK ? smem : base;
        *reinterpret_cast<u32x4 *>(b + off) = v;
    }
    __device__ __forceinline__ void stage_rows(int slot, RowsF &f, const Ptrs &Pn, const Seg &c, int nvalid_n,
                                               const LOffs &o) const
    {
        const unsigned b = (unsigned)(nvalid_n * c.qks * 2);
        const __amdgpu_buffer_rsrc_t r[4] = {rsrc(Pn.k, b), rsrc(Pn.q, b), rsrc(Pn.kn, b), rsrc(Pn.qn, b)};
#pragma unroll
        for (int u = 0; u < OPS; ++u)
#pragma unroll
            for (int si = 0; si < 4; ++si) {
                st16(smem + slot * RING_B + si * ROWS_B, o.rl[u], to_operand<In, E>(f.c[si][u]));
                f.c[si][u] = bload(r[si], o.rg[u]);
            }
    }
    __device__ __forceinline__ void stage_v(int p, VF &f, const Ptrs &Pn, const Seg &c, int nvalid_n,
                                            const LOffs &o) const
    {
        const unsigned b = (unsigned)(nvalid_n * c.vst * 2);
        const __amdgpu_buffer_rsrc_t r0 = rsrc(Pn.v, b), r1 = rsrc(Pn.vn, b);
#pragma unroll
        for (int u = 0; u < VPL; ++u) {
            st16(smem + OFF_VS + p * VSET_B, o.vl[u], f.c[u]);
            f.c[u] = bload(o.vm[u] ? r1 : r0, o.vg[u]);
        }
    }

    // ------------------------------------------------------------------ U: the records
    // U0 (STREAM 0): gates, T, P of the clean block in ring slot `slot`; U1: T~, R.
    template <int STREAM>
    __device__ __forceinline__ void u_record(int slot, int p, float gv, float bv, const QOffs<DK> &qo,
                                             const ut::Consts &us_) const
    {
        const int g = lane >> 4, n = lane & 15;
        float *Gs = us(STREAM), *Bs = Gs + 64;
        const float x = ut::scan32(lane < LP ? gv * kLog2e : 0.f, lane);
        const float gl = ut::lane_value(x, LP - 1);
        Gs[lane] = x;
        Bs[lane] = bv;
        if (lane < LP) {
            if (STREAM == 0) {
                fac(p, 0)[lane] = fexp2(x);
                fac(p, 1)[lane] = fexp2(gl - x);
                fac(p, 2)[lane] = x;
            } else {
                fac(p, 3)[lane] = fexp2(x);
                fac(p, 4)[lane] = fexp2(gl - x);
            }
        }
        const E *K = rows(slot, STREAM == 0 ? 0 : 2);
        const E *Q = rows(slot, STREAM == 0 ? 1 : 3);
        {
            QE kq[NB][DKB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) ld_q<DKB, DK>(kq[rb], K + 16 * rb * DK, qo.q);
            ut::solve_t<NB, DKB>(kq, Gs, Bs, mat(p, STREAM), TS, us_, lane);
        }
        // P (clean, causal) or R (noisy, block end) from the transposed tiles
        // acc = K Q^T: lane (g, n) holds k_(16 bc + 4g + i) . q_(16 br + n), i.e. entry
        // (16 br + n, 16 bc + 4g + i) of Q K^T, four consecutive entries of one row.
        E *M = mat(p, STREAM == 0 ? 2 : 3);
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        f32x4 gc4[NB];
        float grn[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            gc4[b] = ld4f(Gs + 16 * b + 4 * g);
            grn[b] = Gs[16 * b + n];
        }
#pragma unroll
        for (int br = 0; br < NB; ++br) {
            QE qq[DKB];
            ld_q<DKB, DK>(qq, Q + 16 * br * DK, qo.q);
#pragma unroll
            for (int bc = 0; bc < NB; ++bc) {
                f32x4 v = z;
                if (STREAM == 1 || bc <= br) {
                    QE kq[DKB];   // reloaded: keeping the key quads across the solve costs registers
                    ld_q<DKB, DK>(kq, K + 16 * bc * DK, qo.q);
                    const f32x4 kqt = mma_q<E, DKB>(z, kq, qq);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (STREAM == 0) {
                            const bool on = bc < br || 4 * g + i <= n;
                            v[i] = on ? fexp2(-fabsf(grn[br] - gc4[bc][i])) * kqt[i] : 0.f;
                        } else {
                            v[i] = fexp2(-fabsf(gl - gc4[bc][i])) * kqt[i];
                        }
                    }
                }
                st_quad(M + (16 * br + n) * TS + 16 * bc + 4 * g, quad_of<E>(v));
            }
        }
    }
    template <int STREAM>
    __device__ __forceinline__ void u_loop(const Seg &c, const QOffs<DK> &qo) const
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
        u_record<STREAM>(0, 0, lane < LP ? gx : 0.f, lane < LP ? bx : 0.f, qo, usv);
        lds_barrier();
        for (int j = 0; j < c.nb; ++j) {
            load_gates(j + 2, gx, bx);
            u_record<STREAM>((j + 1) % 3, (j + 1) & 1, lane < LP ? gy : 0.f, lane < LP ? by : 0.f, qo, usv);
            gy = gx;
            by = bx;
            lds_barrier();
        }
    }

    // ------------------------------------------------------------------ C: one block
    __device__ __forceinline__ void c_block(int slot, int p, int c0, f32x4 (&S)[DKB], QE (&sq)[DKB], Out *o, Out *on,
                                            int stride, int nvalid, float scale, const QOffs<DK> &qo) const
    {
        const int g = lane >> 4, n = lane & 15;
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        // clean: Delta = T (V - diag(eG) K S0)
        QE dlq[NB], uq[NB];
        {
            f32x4 x[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE kq[DKB];
                ld_q<DKB, DK>(kq, rows(slot, 0) + 16 * rb * DK, qo.q);
                x[rb] = mma_q<E, DKB>(z, kq, sq);
            }
            const In *V = vs(p, 0);
            const float *eG = fac(p, 0);
            QE dq[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                const int r = 16 * rb + 4 * g;
                const f32x4 gq = ld4f(eG + r);
                f32x4 d;
#pragma unroll
                for (int i = 0; i < 4; ++i) d[i] = to_f(V[(r + i) * VS + c0 + n]) - gq[i] * x[rb][i];
                dq[rb] = quad_of<E>(d);
            }
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE tq[NB];
                ld_quads<E, NB>(tq, mat(p, 0) + 16 * rb * TS, TS, lane);
                const f32x4 dl = mma_q<E, NB>(z, tq, dq);
                dlq[rb] = quad_of<E>(dl);
                uq[rb] = quad_of<E>(dl * ld4f(fac(p, 1) + 16 * rb + 4 * g));
            }
        }
        // clean outputs: O = diag(eG) Q S0 + P Delta
        {
            f32x4 acc[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE qq[DKB];
                ld_q<DKB, DK>(qq, rows(slot, 1) + 16 * rb * DK, qo.q);
                const f32x4 x2 = mma_q<E, DKB>(z, qq, sq) * ld4f(fac(p, 0) + 16 * rb + 4 * g);
                QE pq[NB];
                ld_quads<E, NB>(pq, mat(p, 2) + 16 * rb * TS, TS, lane);
                acc[rb] = mma_q<E, NB>(x2, pq, dlq);
            }
            store_out<Out, NB>(o, stride, nvalid, c0, acc, scale, lane);
        }
        // noisy: Delta~ = T~ (V~ - diag(eG~) K~ S0), O~ = gamma~_n Q~ S0 + R Delta~
        {
            f32x4 x3[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE kq[DKB];
                ld_q<DKB, DK>(kq, rows(slot, 2) + 16 * rb * DK, qo.q);
                x3[rb] = mma_q<E, DKB>(z, kq, sq);
            }
            const In *V = vs(p, 1);
            const float *eG = fac(p, 3);
            QE dq[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                const int r = 16 * rb + 4 * g;
                const f32x4 gq = ld4f(eG + r);
                f32x4 d;
#pragma unroll
                for (int i = 0; i < 4; ++i) d[i] = to_f(V[(r + i) * VS + c0 + n]) - gq[i] * x3[rb][i];
                dq[rb] = quad_of<E>(d);
            }
            QE nq[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE tq[NB];
                ld_quads<E, NB>(tq, mat(p, 1) + 16 * rb * TS, TS, lane);
                nq[rb] = quad_of<E>(mma_q<E, NB>(z, tq, dq));
            }
            const float gn_end = eG[LP - 1];
            f32x4 acc[NB];
#pragma unroll
            for (int rb = 0; rb < NB; ++rb) {
                QE qq[DKB];
                ld_q<DKB, DK>(qq, rows(slot, 3) + 16 * rb * DK, qo.q);
                const f32x4 x4 = mma_q<E, DKB>(z, qq, sq) * gn_end;
                QE rq[NB];
                ld_quads<E, NB>(rq, mat(p, 3) + 16 * rb * TS, TS, lane);
                acc[rb] = mma_q<E, NB>(x4, rq, nq);
            }
            store_out<Out, NB>(on, stride, nvalid, c0, acc, scale, lane);
        }
        // state: S <- gamma_n S0 + K^T diag(dG) Delta
        const float decay = fac(p, 0)[LP - 1];
        const E *K = rows(slot, 0);
#pragma unroll
        for (int kb = 0; kb < DKB; ++kb) {
            QE kt[NB];
            kt_quads<NB, DK>(kt, K, kb, qo);
            S[kb] = mma_q<E, NB>(S[kb] * decay, kt, uq);
            sq[kb] = quad_of<E>(S[kb]);
        }
    }

    // ------------------------------------------------------------------ the segment
    __device__ void run(const Seg &c) const
    {
        const int nb = c.nb;
        QOffs<DK> qo;
        if (wave < NC) {
            qo.make(lane);
            // ---- C
            const int g = lane >> 4, n = lane & 15;
            const int c0 = 16 * wave;
            f32x4 S[DKB];
            QE sq[DKB];
#pragma unroll
            for (int kb = 0; kb < DKB; ++kb) {
                f32x4 s = {0.f, 0.f, 0.f, 0.f};
                if (c.s0) {
                    const float *src = c.s0 + (long)(16 * kb + 4 * g) * c.dv + c0 + n;
#pragma unroll
                    for (int i = 0; i < 4; ++i) s[i] = src[i * c.dv];
                }
                S[kb] = s;
                sq[kb] = quad_of<E>(s);
            }
            Ptrs pc = c.p0;
            lds_barrier();
            lds_barrier();
            for (int j = 0; j < nb; ++j) {
                c_block(j % 3, j & 1, c0, S, sq, pc.o, pc.on, c.vst, nvalid_of(c, j), c.scale, qo);
                advance(pc, c);
                lds_barrier();
            }
            if (c.ht) {
#pragma unroll
                for (int kb = 0; kb < DKB; ++kb) {
                    float *dst = c.ht + (long)(16 * kb + 4 * g) * c.dv + c0 + n;
#pragma unroll
                    for (int i = 0; i < 4; ++i) dst[i * c.dv] = S[kb][i];
                }
            }
        } else if (wave == NC) {
            qo.make(lane);
            u_loop<0>(c, qo);
        } else if (wave == NC + 1) {
            qo.make(lane);
            u_loop<1>(c, qo);
        } else {
            // ---- L: step j stages the rows of block j + 2 and V of block j + 1, each
            // refilled from two blocks further on
            const int tw = wave - NC - 2;
            LOffs o;
            make_loffs(c, tw, o);
            auto nv = [&](int jj) { return nvalid_of(c, jj); };
            Ptrs pr = c.p0, pv = c.p0;
            RowsF r0, r1;
            VF v0, v1;
            fetch_rows(pr, c, nv(0), o, r0);
            advance(pr, c);
            fetch_rows(pr, c, nv(1), o, r1);
            advance(pr, c);
            fetch_v(pv, c, nv(0), o, v0);
            advance(pv, c);
            fetch_v(pv, c, nv(1), o, v1);
            advance(pv, c);
            stage_rows(0, r0, pr, c, nv(2), o);
            advance(pr, c);
            stage_rows(1, r1, pr, c, nv(3), o);
            advance(pr, c);
            stage_v(0, v0, pv, c, nv(2), o);
            advance(pv, c);
            lds_barrier();
            lds_barrier();
            int j = 0;
            for (; j + 1 < nb; j += 2) {
                stage_rows((j + 2) % 3, r0, pr, c, nv(j + 4), o);
                advance(pr, c);
                stage_v(1, v1, pv, c, nv(j + 3), o);
                advance(pv, c);
                lds_barrier();
                stage_rows((j + 3) % 3, r1, pr, c, nv(j + 5), o);
                advance(pr, c);
                stage_v(0, v0, pv, c, nv(j + 4), o);
                advance(pv, c);
                lds_barrier();
            }
            if (j < nb) {
                stage_rows((j + 2) % 3, r0, pr, c, 0, o);
                stage_v(1, v1, pv, c, 0, o);
                lds_barrier();
            }
        }
    }
};

// One workgroup's (chain, segment) of the out kernel from its block id.
template <typename K>
__device__ __forceinline__ void run_segment(const ChunkArgs &a, unsigned char *smem)
{
    typedef typename K::Seg Seg;
    typedef typename K::Ptrs Ptrs;
    constexpr int DK = K::DK_;
    // Workgroups come in groups of (position in order, segment, q/k head); a group's members
    // are its v-heads times the d_v tiles, all reading the same q/k rows.  Eight groups
    // interleave, so that the members of a group have ids congruent mod 8 and run on one
    // XCD (workgroup ids are dealt to the eight XCDs in turn).
    const int r_v = a.h_v / a.h_qk, M = r_v * a.n_ot;
    const int u = blockIdx.x, blk = u / (8 * M), rem = u % (8 * M);
    const int grp = blk * 8 + rem % 8, mem = rem / 8;
    if (grp >= a.n_groups) return;
    int pos, s, hq;
    if (a.cu) {
        // binary search for the last position whose segments-before * h_qk <= grp
        int lo = 0, hi = a.n_order - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((long)segs_before(a, mid) * a.h_qk <= grp) lo = mid; else hi = mid - 1;
        }
        pos = lo;
        const int r = grp - segs_before(a, pos) * a.h_qk;
        s = r / a.h_qk;
        hq = r % a.h_qk;
    } else {
        const int per = nseg_of(a.nblk, a.G) * a.h_qk;
        pos = grp / per;
        const int r = grp % per;
        s = r / a.h_qk;
        hq = r % a.h_qk;
    }
    const int h = hq * r_v + mem / a.n_ot, v0 = (mem % a.n_ot) * K::DV;
    const Geo geo = geo_of(a, pos);
    if (s >= geo.nseg) return;
    const long row0 = geo.base + (long)s * a.G * a.L;
    Seg c;
    const long qk_off = (row0 * a.h_qk + hq) * DK;
    const long v_off = (row0 * a.h_v + h) * a.dv + v0;
    const long g_off = row0 * a.h_v + h;
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
    c.p0.o = static_cast<typename K::OutT *>(a.o) + v_off;
    c.p0.on = static_cast<typename K::OutT *>(a.on) + v_off;
    c.qks = a.h_qk * DK;
    c.vst = a.h_v * a.dv;
    c.gst = a.h_v;
    c.qk_blk = (long)a.L * c.qks;
    c.v_blk = (long)a.L * c.vst;
    c.g_blk = (long)a.L * c.gst;
    c.len = geo.len - (long)s * a.G * a.L;
    const int left = geo.nb - s * a.G;
    c.nb = left < a.G ? left : a.G;
    c.L = a.L;
    const long st_off = ((long)geo.doc * a.h_v + h) * DK * a.dv + v0;
    if (s == 0)
        c.s0 = a.h0 ? a.h0 + st_off : nullptr;
    else
        c.s0 = a.ckpt + ckpt_index(a, pos, h, geo.nseg, s) * DK * a.dv + v0;
    c.ht = (a.ht && s == geo.nseg - 1) ? a.ht + st_off : nullptr;
    c.dv = a.dv;
    c.scale = a.scale;
    K k(smem);
    k.run(c);
}

}  // namespace chunked

}  // namespace bdgdn
