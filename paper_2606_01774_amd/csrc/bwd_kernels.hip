// bwd_kernels.hip -- backward of the two-stream training forward (Appendix "Backward
// primitives": the block-level chain rule eq. dh-block-recursion, the noisy block-end
// readout backward eq. noisy-readout-bwd, and the clean chunk backward), for gfx950.
//
// The per-step backward of the paper (eq. per-step-bwd) needs every per-step state; here
// each block is differentiated in its block (WY) form instead, which needs only the
// block's seed state S0.  For one block of n positions from S0, with local cumulative
// log-gates G (gamma = exp G, gamma_n the last), D_i = gamma_n / gamma_i and
//   A_ri = beta_r (gamma_r/gamma_i) k_r.k_i (i < r),  M = (I + A)^-1,  T = M diag(beta),
//   X = K S0,  R = V - Gamma X,  Delta = T R,  S_n = gamma_n S0 + K^T D Delta,
//   clean:  O = s (Gamma Q S0 + P Delta),  P = Q K^T o Mc,  Mc_ri = gamma_r/gamma_i (i <= r)
//   noisy:  O~ = s Q S_n  (every position reads the block-end state),
// and the gradient dS_n of the block-end state (clean: the gradient arriving from the later
// blocks; noisy: s Q^T dO~), the backward is
//   E = dO Delta^T,  dDelta = [clean] s P^T dO + D K dS_n,  dR = T^T dDelta = dV,
//   dQ = [clean] s Gamma dO S0^T + (s E o Mc) K   |  [noisy] s gamma_n dO S0^T + s (E D) K,
//   dK = [clean] (s E o Mc)^T Q + D Delta dS_n^T - Gamma dR S0^T + (dKK + dKK^T) K,
//   dT = dDelta R^T,  dbeta_i = sum_r dT_ri M_ri + sum_i' dA_ii' F_ii',
//   dA = strictly lower part of -M^T (dT diag beta) M^T,  dKK_ri = dA_ri beta_r gamma_r/gamma_i,
//   dS0 = gamma_n dS_n + [clean] s Q^T Gamma dO - K^T Gamma dR,
// with the gate gradients collected on the local cumulative gates (dG) and dg = the
// reverse cumulative sum of dG inside the block.  The chain rule across blocks:
// dh_(b-1) = dS0(clean block b) + dS0(noisy block b), since the noisy block b is seeded with
// the clean state at the end of block b - 1.
//
// Three phases after the clean scan has written every block's seed (launch_scan_states, fp16):
//  1. every noisy block in parallel: its gradients and its seed's gradient, plus the part of
//     the clean block at the same position that does not depend on the state gradient dh
//     (clean_prep); their sum c_b is the dh-independent part of dh_(b-1);
//  2. the reverse scan of the clean state gradient over the blocks of each (sequence,
//     v-head), in 32-column tiles (the columns are independent):
//     dh_(b-1) = gamma_n dh_b + c_b - K^T (U K) dh_b with U = Gamma T^T D from phase 1;
//  3. every clean block in parallel from its seed and the gradient at its end.
// In time segments (BwdArgs::seg; the strided clean checkpoints of the checkpoint build) the
// same three phases run over one segment of every chain at a time, last segment first: the
// seeds come from the segment's checkpoint, the scan starts from the gradient the later
// segment left in the carry and leaves its own there, and the units are numbered inside the
// segment by the segment tables (bdgdn_bwd_seg_plan_kernel).
// Products are MFMA tiles on fp16 operands with fp32 accumulation: k-contiguous operands by
// 16-byte LDS reads, the others by the LDS transpose load, and results that are the next
// product's operand kept in registers; M = (I + A)^-1 by the register-resident doubling solve
// (ut::solve_t), the dA products in fp32 MFMA.  Blocks are padded to 32 positions with
// identity steps (k = 0, beta = 0, g = 0), which change nothing.
#include "common.hpp"
#include "bwd.hpp"
#include "kernels.hpp"
#include "ut.hpp"

namespace bdgdn {

namespace {

constexpr int NP = 32;           // positions per (padded) block
constexpr int DD = 128;          // d_k = d_v
constexpr int LDH = DD + 8;      // f16 row stride of [*][128] LDS matrices
constexpr int LDF = NP + 1;      // fp32 row stride of [32][32] LDS matrices
constexpr int LDM = NP + 8;      // f16 row stride of [32][32] LDS matrices
constexpr int kWaves = 8;

struct Smem {
    _Float16 S0[DD * LDH];       // seed state (d_k x d_v)
    _Float16 dS[DD * LDH];       // dS_n (d_k x d_v)
    _Float16 Q[NP * LDH], K[NP * LDH], R[NP * LDH], dO[NP * LDH];
    _Float16 Dl[NP * LDH], dDl[NP * LDH];
    _Float16 dR[NP * LDH];       // -Gamma dR
    _Float16 Mh[NP * LDM];       // M = (I + A)^-1
    _Float16 Ph[NP * LDM];       // clean: P = (Q K^T) o Mc
    _Float16 dPh[NP * LDM];      // the gradient of Q K^T: clean s E o Mc, noisy s E_ri D_i
    _Float16 Wh[NP * LDM];       // dKK + dKK^T (clean_prep: U)
    float KK[NP * LDF], dT[NP * LDF], W[NP * LDF];
    float TdA[NP * LDF];         // T (T_ci = M_ci beta_i at [c][i]), later dA
    float Mt[NP * LDF];          // M^T (fp32)
    float G[NP], G2[NP], gam[NP], bet[NP], dB[NP];   // G2: cumulative log2-gates
    // the gradient of the local cumulative gates, as per-wave partial sums: every
    // contribution goes to the row of the wave that makes it, and the rows are added in a
    // fixed order at the end (deterministic, unlike float atomics from several waves)
    float part[kWaves][NP];
};
static_assert(sizeof(Smem) <= 160 * 1024, "one workgroup's LDS");

typedef __fp16 fp16x4_t __attribute__((__vector_size__(4 * sizeof(__fp16))));

// Operands of v_mfma_f32_16x16x16f16, lane (g, n) = (lane / 16, lane % 16): A row n with
// k = 4 g .. 4 g + 3, B column n with the same k, C column n with rows 4 g .. 4 g + 3.  A C
// tile kept in registers is therefore the B operand of a product contracting over its rows.
//
// A from a row-major matrix with k contiguous (one 8-byte read).
__device__ __forceinline__ f16x4 op_row(const _Float16 *X, int ld, int m0, int k0, int lane)
{
    return *reinterpret_cast<const f16x4 *>(X + (m0 + (lane & 15)) * ld + k0 + 4 * (lane >> 4));
}
// X[k0 + 4 g + e][c0 + n] of a row-major matrix: the B operand X (k = row) or the A operand
// X^T, by the LDS transpose load ds_read_b64_tr_b16 (lane L reads the 8 bytes at row
// k0 + L / 4, columns c0 + 4 (L % 4); each 16-lane group receives the columns of the 4 x 16
// block its lanes read).
__device__ __forceinline__ f16x4 op_tr(const _Float16 *X, int ld, int k0, int c0, int lane)
{
    const _Float16 *p = X + (k0 + (lane >> 2)) * ld + c0 + 4 * (lane & 3);
    return __builtin_bit_cast(f16x4, __builtin_amdgcn_ds_read_tr16_b64_v4f16(
                                         (__attribute__((address_space(3))) fp16x4_t *)(p)));
}
__device__ __forceinline__ f32x4 mfma(f16x4 a, f16x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f16x4 h4(f32x4 v)
{
    return f16x4{(_Float16)v[0], (_Float16)v[1], (_Float16)v[2], (_Float16)v[3]};
}
__device__ __forceinline__ f16x4 scale4(f16x4 v, f32x4 f)
{
    return f16x4{(_Float16)((float)v[0] * f[0]), (_Float16)((float)v[1] * f[1]), (_Float16)((float)v[2] * f[2]),
                 (_Float16)((float)v[3] * f[3])};
}
__device__ __forceinline__ f32x4 ld4(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }

__device__ __forceinline__ float ex(float x) { return __expf(x); }

// v added to *dst (LDS) atomically.
__device__ __forceinline__ void lds_add(float *dst, float v) { atomicAdd(dst, v); }

// Sum over the 16 lanes of each lane row (the columns of a C tile row), by DPP row shifts:
// valid in lane 15 of the row.
__device__ __forceinline__ float row_total(float v)
{
    v += ut::dpp<0x111>(v);
    v += ut::dpp<0x112>(v);
    v += ut::dpp<0x114>(v);
    v += ut::dpp<0x118>(v);
    return v;
}
// Sums over lanes 0 .. 31 and 32 .. 63, each returned to the lanes of its half.
__device__ __forceinline__ float half_total(float v, int lane)
{
    const float t = row_total(v);
    const float h0 = ut::lane_value(t, 15) + ut::lane_value(t, 31);
    const float h1 = ut::lane_value(t, 47) + ut::lane_value(t, 63);
    return lane < 32 ? h0 : h1;
}
__device__ __forceinline__ float wave_total(float v)
{
    const float t = row_total(v);
    return (ut::lane_value(t, 15) + ut::lane_value(t, 31)) + (ut::lane_value(t, 47) + ut::lane_value(t, 63));
}

// One thread's share of a 32 x 128 row block (row tid / 16, the 8 values from 8 (tid % 16)),
// loaded into registers ahead of its store to LDS as fp16, so that all loads of a unit are
// in flight together.
template <typename In> struct Row8;
template <> struct Row8<__bf16> {
    bf16x8 v;
    __device__ __forceinline__ void load(const __bf16 *p) { v = *reinterpret_cast<const bf16x8 *>(p); }
    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (__bf16)0.f;
    }
    __device__ __forceinline__ f16x8 h(float sg = 1.f) const
    {
        f16x8 r;
#pragma unroll
        for (int j = 0; j < 8; ++j) r[j] = (_Float16)((float)v[j] * sg);
        return r;
    }
};
template <> struct Row8<float> {
    f32x4 lo, hi;
    __device__ __forceinline__ void load(const float *p)
    {
        lo = ld4(p);
        hi = ld4(p + 4);
    }
    __device__ __forceinline__ void zero() { lo = hi = f32x4{0.f, 0.f, 0.f, 0.f}; }
    __device__ __forceinline__ f16x8 h(float sg = 1.f) const
    {
        f16x8 r;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            r[j] = (_Float16)(lo[j] * sg);
            r[4 + j] = (_Float16)(hi[j] * sg);
        }
        return r;
    }
};
template <typename In> __device__ __forceinline__ Row8<In> load_rows(const In *src, long stride, int nvalid, int tid)
{
    const int r = tid >> 4, c = (tid & 15) * 8;
    Row8<In> x;
    if (r < nvalid)
        x.load(src + (long)r * stride + c);
    else
        x.zero();
    return x;
}
template <typename In> __device__ __forceinline__ void store_rows(_Float16 *dst, const Row8<In> &x, int tid,
                                                                  float sg = 1.f)
{
    const int r = tid >> 4, c = (tid & 15) * 8;
    *reinterpret_cast<f16x8 *>(dst + r * LDH + c) = x.h(sg);
}

// The fp16 seed state (128 x 128, 32 KB): four 16-byte pieces per thread.
struct SeedRegs {
    f16x8 v[4];
};
__device__ __forceinline__ SeedRegs load_seed(const _Float16 *src, int tid)
{
    SeedRegs x;
#pragma unroll
    for (int it = 0; it < 4; ++it) x.v[it] = *reinterpret_cast<const f16x8 *>(src + (tid + 512 * it) * 8);
    return x;
}
__device__ __forceinline__ void store_seed(_Float16 *dst, const SeedRegs &x, int tid)
{
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int e = (tid + 512 * it) * 8;
        *reinterpret_cast<f16x8 *>(dst + (e / DD) * LDH + e % DD) = x.v[it];
    }
}
// The same 128 x 128 fp16 state stored tile-native (64 tiles of 16 x 16 in row-major tile
// order, each lane-major in the MFMA result layout: lane 16 g + r holds rows 4 g .. 4 g + 3
// of column r), loaded by load_seed as 16-byte chunks (two lanes of one tile each), into
// the row-major LDS copy.
__device__ __forceinline__ void store_tiles(_Float16 *dst, const SeedRegs &x, int tid)
{
#pragma unroll
    for (int it = 0; it < 4; ++it)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int vec = 2 * (tid + 512 * it) + hh, tile = vec >> 6, ln = vec & 63;
            _Float16 *d = dst + (16 * (tile >> 3) + 4 * (ln >> 4)) * LDH + 16 * (tile & 7) + (ln & 15);
#pragma unroll
            for (int j = 0; j < 4; ++j) d[j * LDH] = x.v[it][4 * hh + j];
        }
}

// Block-local cumulative log-gates G (and G2 = G log2 e) and gamma = exp G, by wave 0 (a
// 32-lane scan of the staged gates in G).
__device__ __forceinline__ void cum_gates(Smem &sm, int lane)
{
    float x = lane < NP ? sm.G[lane] : 0.f;
#pragma unroll
    for (int o = 1; o < NP; o <<= 1) {
        const float y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane < NP) {
        sm.G[lane] = x;
        sm.G2[lane] = x * kLog2e;
        sm.gam[lane] = ex(x);
    }
}

// M = (I + A)^-1 of the staged block into sm.Mh, by the register-resident doubling solve of
// one wave (ut::solve_t) from the keys K (LDS, [32][LDH]) and the gates sm.G2, sm.bet.
__device__ __forceinline__ void solve_m(Smem &sm, const _Float16 *K, int lane)
{
    ut::QE kq[2][DD / 16];
    const int r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int kb = 0; kb < DD / 16; ++kb)
            kq[rb][kb] = *reinterpret_cast<const f16x4 *>(K + (16 * rb + r) * LDH + 16 * kb + 4 * g);
    ut::Consts cs;
    ut::make_consts(cs, lane);
    ut::solve_t<2, DD / 16, false>(kq, sm.G2, sm.bet, sm.Mh, LDM, cs, lane);
}

// T^T operand quads of row block tm: A(m = i, k = r) = T_ri = M_ri beta_i for r in 0 .. 31
// (M^T by the transpose load, scaled by beta of the row i = 16 tm + n).
__device__ __forceinline__ void tt_ops(const Smem &sm, int tm, int lane, f16x4 &t0, f16x4 &t1)
{
    const float b = sm.bet[16 * tm + (lane & 15)];
    const f32x4 bb = {b, b, b, b};
    t0 = scale4(op_tr(sm.Mh, LDM, 0, 16 * tm, lane), bb);
    t1 = scale4(op_tr(sm.Mh, LDM, 16, 16 * tm, lane), bb);
}

struct StreamPtrs {
    const __bf16 *q, *k, *v;   // first row of the block (q/k head hq, v head h)
    const float *g, *beta;     // first row (head h), stride h_v
    const void *dout;          // first row (head h)
    float *dq, *dk, *dv, *dg, *db;   // first row of the gradients
};

// A block's inputs in registers (V only with WITH_V); g, b: the gate and step size of
// position tid (tid < 32).
template <typename Od, bool WITH_V> struct BlockRows {
    Row8<__bf16> q, k, v;
    Row8<Od> dout;
    float g, b;
};
template <typename Od, bool WITH_V>
__device__ __forceinline__ BlockRows<Od, WITH_V> load_block(const StreamPtrs &p, int h_qk, int h_v, int nvalid, int tid)
{
    const long qks = (long)h_qk * DD, vs = (long)h_v * DD;
    BlockRows<Od, WITH_V> x;
    x.q = load_rows(p.q, qks, nvalid, tid);
    x.k = load_rows(p.k, qks, nvalid, tid);
    if constexpr (WITH_V) x.v = load_rows(p.v, vs, nvalid, tid);
    x.dout = load_rows(static_cast<const Od *>(p.dout), vs, nvalid, tid);
    const bool ok = tid < NP && tid < nvalid;
    x.g = ok ? p.g[(long)tid * h_v] : 0.f;
    x.b = ok ? p.beta[(long)tid * h_v] : 0.f;
    return x;
}

}  // namespace

// q/k gradient x into *dst: stored for the first v-head of a q/k head, added for the others
// (a workgroup runs the v-heads of a q/k head one after the other, and the same thread
// writes the same element for each, so the sum has a fixed order; see unit_of).
__device__ __forceinline__ void put_qk(bool add, float *dst, float x)
{
    if (add)
        *dst += x;
    else
        *dst = x;
}

// What block_bwd differentiates: a clean block (per-position outputs, dS_n given), a noisy
// block (every position reads the block-end state, dS_n = s Q^T dO formed here), or a block
// with no outputs of its own whose dS_n is given (the sub-blocks of a noisy block of two,
// whose readout gradient the caller has formed).
enum class Mode { Clean, Noisy, Given };

// One block's gradients.  S0 (LDS f16) holds the seed.  For Clean and Given dS (LDS, f16)
// holds dS_n on entry; for Noisy dS_n is formed here from the block-end readout.  Noisy and
// Given add the seed's gradient dS0 into acc (registers, the C-tile layout of a state
// gradient: wave w holds column block w, row blocks 0 .. 7).  Wave w computes the 16 columns 16 w .. 16 w + 15 of every 32 x 128 and 128 x 128
// product.  hook1() runs once the arrays R, dDl and dO are dead (after the dR / dQ phase),
// hook2() two phases later: a persistent caller loads the next unit's clean rows in the one
// and stages them into those arrays in the other.
template <Mode MODE, typename Od, typename H1, typename H2>
__device__ __forceinline__ void block_bwd(Smem &sm, const StreamPtrs &p, const BwdArgs &a, int nvalid, const BlockRows<Od, true> &in,
                          float (&acc)[8][4], int tid, bool add_qk, const H1 &hook1, const H2 &hook2)
{
    constexpr bool CLEAN = MODE == Mode::Clean;     // per-position outputs
    constexpr bool READOUT = MODE == Mode::Noisy;   // dS_n from the block-end readout
    constexpr bool SEED = MODE != Mode::Clean;      // the seed's gradient into acc
    constexpr bool DQ = MODE != Mode::Given;        // q gradients of the block's rows
    const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15, c0 = 16 * wave;
    const float s = a.scale;
    const float inv = a.range[1];   // every gradient is linear in the scaled upstream gradients
    const long vs = (long)a.h_v * DD;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    // This lane's shares of the gate gradients that are sums over a row of a 32 x 128 product:
    // rowg[tm][j] for row 16 tm + 4 g + j (this lane's column), dlast for the last position;
    // reduced once, at the end.
    float rowg[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}}, dlast = 0.f;
    // ---- stage rows and gates
    store_rows(sm.Q, in.q, tid);
    store_rows(sm.K, in.k, tid);
    store_rows(sm.R, in.v, tid);   // V, becomes R below
    store_rows(sm.dO, in.dout, tid, a.range[0]);   // upstream gradients times the range scale
    if (tid < NP) {
        sm.bet[tid] = in.b;
        sm.G[tid] = in.g;
        sm.dB[tid] = 0.f;
    }
    if (tid < kWaves * NP) sm.part[tid / NP][tid % NP] = 0.f;
    __syncthreads();
    if (wave == 0) cum_gates(sm, lane);
    __syncthreads();
    const float Gn = sm.G[NP - 1];
    const float gn = ex(Gn);
    // ---- M (wave 0); KK = K K^T and P = (Q K^T) o Mc (clean) (waves 1 .. 4); X = K S0 ->
    // R = V - Gamma X; dS_n (noisy: s Q^T dO) with its share gamma_n dS_n of dS0 and the gate
    // term dG_last += gamma_n <dS_n, S0>
    if (wave == 0) {
        solve_m(sm, sm.K, lane);
    } else if (wave <= 4) {
        const int m0 = 16 * ((wave - 1) >> 1), n0 = 16 * ((wave - 1) & 1);
        f32x4 c = tile_mma<_Float16, DD>(z, sm.K + m0 * LDH, LDH, sm.K + n0 * LDH, LDH, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.KK[(m0 + 4 * g4 + j) * LDF + n0 + rr] = c[j];
        if constexpr (CLEAN) {
            c = tile_mma<_Float16, DD>(z, sm.Q + m0 * LDH, LDH, sm.K + n0 * LDH, LDH, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = m0 + 4 * g4 + j, i = n0 + rr;
                sm.Ph[r * LDM + i] = (_Float16)(i <= r ? c[j] * ex(sm.G[r] - sm.G[i]) : 0.f);
            }
        }
    }
    f16x4 s0q[8];   // S0 tiles (tm, w): the B operands of K S0 and the layout of dS_n
#pragma unroll
    for (int tm = 0; tm < 8; ++tm) s0q[tm] = op_tr(sm.S0, LDH, 16 * tm, c0, lane);
#pragma unroll
    for (int tm = 0; tm < 2; ++tm) {
        f32x4 x = z;
#pragma unroll
        for (int kb = 0; kb < 8; ++kb) x = mfma(op_row(sm.K, LDH, 16 * tm, 16 * kb, lane), s0q[kb], x);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, c = c0 + rr;
            sm.R[r * LDH + c] = (_Float16)((float)sm.R[r * LDH + c] - sm.gam[r] * x[j]);
        }
    }
    f16x4 dsq[8];   // dS_n tiles (tm, w): the B operands of K dS_n
    {
        f16x4 dob[2];
        if constexpr (READOUT) {
            dob[0] = op_tr(sm.dO, LDH, 0, c0, lane);
            dob[1] = op_tr(sm.dO, LDH, 16, c0, lane);
        }
        float wg = 0.f;
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            f32x4 c;
            if constexpr (!READOUT) {   // dS_n tile (tm, w) from LDS by the transpose load
                dsq[tm] = op_tr(sm.dS, LDH, 16 * tm, c0, lane);
#pragma unroll
                for (int j = 0; j < 4; ++j) c[j] = (float)dsq[tm][j];
            } else {
                c = mfma(op_tr(sm.Q, LDH, 16, 16 * tm, lane), dob[1], mfma(op_tr(sm.Q, LDH, 0, 16 * tm, lane), dob[0], z));
                c *= s;
                dsq[tm] = h4(c);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if constexpr (READOUT) sm.dS[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = dsq[tm][j];
                if constexpr (SEED) acc[tm][j] += gn * c[j];
                wg += c[j] * (float)s0q[tm][j];
            }
        }
        dlast += gn * wg;
    }
    __syncthreads();
    // ---- Delta = T R (T_ri = M_ri beta_i); fp32 copies of T and M^T for the dA products
    {
        const f32x4 b0 = ld4(sm.bet + 4 * g4), b1 = ld4(sm.bet + 16 + 4 * g4);
        const f16x4 r0 = op_tr(sm.R, LDH, 0, c0, lane), r1 = op_tr(sm.R, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            const f16x4 t0 = scale4(op_row(sm.Mh, LDM, 16 * tm, 0, lane), b0);
            const f16x4 t1 = scale4(op_row(sm.Mh, LDM, 16 * tm, 16, lane), b1);
            const f32x4 d = mfma(t1, r1, mfma(t0, r0, z));
#pragma unroll
            for (int j = 0; j < 4; ++j) sm.Dl[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = (_Float16)d[j];
        }
    }
    for (int e = tid; e < NP * NP; e += 64 * kWaves) {
        const int r = e / NP, i = e % NP;
        const float m = (float)sm.Mh[r * LDM + i];
        sm.TdA[r * LDF + i] = m * sm.bet[i];
        sm.Mt[i * LDF + r] = m;
    }
    __syncthreads();
    // ---- E = dO Delta^T (waves 0 .. 3), with the gradient of Q K^T into dPh and (clean) the
    // gates of Mc, W = s E o P: dG_r += sum_i W_ri, dG_i -= sum_r W_ri
    if (DQ && wave < 4) {
        const int m0 = 16 * (wave >> 1), n0 = 16 * (wave & 1), i = n0 + rr;
        const f32x4 e4 = tile_mma<_Float16, DD>(z, sm.dO + m0 * LDH, LDH, sm.Dl + n0 * LDH, LDH, lane);
        float colw = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = m0 + 4 * g4 + j;
            if constexpr (CLEAN) {
                const float dec = i <= r ? ex(sm.G[r] - sm.G[i]) : 0.f;
                sm.dPh[r * LDM + i] = (_Float16)(s * e4[j] * dec);
                const float w = s * e4[j] * (float)sm.Ph[r * LDM + i];
                if (wave >> 1)
                    rowg[1][j] += w;
                else
                    rowg[0][j] += w;
                colw += w;
            } else {
                sm.dPh[r * LDM + i] = (_Float16)(s * e4[j] * ex(Gn - sm.G[i]));
            }
        }
        if constexpr (CLEAN) {
            colw += __shfl_xor(colw, 16);
            colw += __shfl_xor(colw, 32);
            if (g4 == 0) lds_add(&sm.part[wave][i], -colw);
        }
    }
    // dDelta = [clean] s P^T dO + D K dS_n, with the D-term gate gradient
    // w_r = D_r sum_c (K dS_n)_rc Delta_rc: dG_last += w, dG_r -= w
    {
        f16x4 do0, do1;
        if constexpr (CLEAN) {
            do0 = op_tr(sm.dO, LDH, 0, c0, lane);
            do1 = op_tr(sm.dO, LDH, 16, c0, lane);
        }
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            f32x4 kds = z;
#pragma unroll
            for (int kb = 0; kb < 8; ++kb) kds = mfma(op_row(sm.K, LDH, 16 * tm, 16 * kb, lane), dsq[kb], kds);
            f32x4 pd = z;
            if constexpr (CLEAN)
                pd = mfma(op_tr(sm.Ph, LDM, 16, 16 * tm, lane), do1, mfma(op_tr(sm.Ph, LDM, 0, 16 * tm, lane), do0, z));
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, c = c0 + rr;
                const float Dr = ex(Gn - sm.G[r]);
                sm.dDl[r * LDH + c] = (_Float16)(s * pd[j] + Dr * kds[j]);
                const float w = Dr * kds[j] * (float)sm.Dl[r * LDH + c];
                rowg[tm][j] -= w;
                dlast += w;
            }
        }
    }
    __syncthreads();
    // ---- dR = T^T dDelta (= dV), kept as -Gamma dR (LDS and, as B operands, registers);
    // [noisy, given] dS0 += K^T (-Gamma dR); dQ; dT = dDelta R^T (waves 4 .. 7)
    f16x4 drq[2];
    {
        const f16x4 dd0 = op_tr(sm.dDl, LDH, 0, c0, lane), dd1 = op_tr(sm.dDl, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            f16x4 t0, t1;
            tt_ops(sm, tm, lane, t0, t1);
            const f32x4 c = mfma(t1, dd1, mfma(t0, dd0, z));
            f32x4 ng;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, col = c0 + rr;
                if (r < nvalid) p.dv[(long)r * vs + col] = c[j] * inv;
                ng[j] = -sm.gam[r] * c[j];
            }
            drq[tm] = h4(ng);
#pragma unroll
            for (int j = 0; j < 4; ++j) sm.dR[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = drq[tm][j];
        }
    }
    if constexpr (SEED) {
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            const f32x4 c =
                mfma(op_tr(sm.K, LDH, 16, 16 * tm, lane), drq[1], mfma(op_tr(sm.K, LDH, 0, 16 * tm, lane), drq[0], z));
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[tm][j] += c[j];
        }
    }
    if constexpr (DQ) {   // dQ = [clean] s Gamma (dO S0^T) + dPh K  |  [noisy] s gamma_n (dO S0^T) + dPh K
        const f16x4 k0q = op_tr(sm.K, LDH, 0, c0, lane), k1q = op_tr(sm.K, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            f32x4 c = tile_mma<_Float16, DD>(z, sm.dO + 16 * tm * LDH, LDH, sm.S0 + c0 * LDH, LDH, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, col = c0 + rr;
                if constexpr (CLEAN) {
                    // gate term of Gamma Q S0: dG_r += s gamma_r sum_a Q_ra (dO S0^T)_ra
                    rowg[tm][j] += s * sm.gam[r] * c[j] * (float)sm.Q[r * LDH + col];
                    c[j] *= s * sm.gam[r];
                } else {
                    c[j] *= s * gn;
                }
            }
            c = mfma(op_row(sm.dPh, LDM, 16 * tm, 16, lane), k1q, mfma(op_row(sm.dPh, LDM, 16 * tm, 0, lane), k0q, c));
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, col = c0 + rr;
                if (r < nvalid) put_qk(add_qk, p.dq + (long)r * a.h_qk * DD + col, c[j] * inv);
            }
        }
    }
    if (wave >= 4) {
        const int m0 = 16 * ((wave - 4) >> 1), n0 = 16 * ((wave - 4) & 1);
        const f32x4 c = tile_mma<_Float16, DD>(z, sm.dDl + m0 * LDH, LDH, sm.R + n0 * LDH, LDH, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.dT[(m0 + 4 * g4 + j) * LDF + n0 + rr] = c[j];
    }
    __syncthreads();
    hook1();   // R, dDl, dO are dead from here on
    // ---- dbeta, dA = strictly lower part of -M^T (dT diag beta) M^T (fp32 MFMA)
    // W = dT T^T (W_rc = sum_i dT_ri beta_i M_ci), stored transposed; dbeta_i += sum_r dT_ri M_ri
    if (wave < 4) {
        const int m0 = 16 * (wave >> 1), n0 = 16 * (wave & 1);
        const f32x4 c = tile_mma<float, NP>(z, sm.dT + m0 * LDF, LDF, sm.TdA + n0 * LDF, LDF, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.W[(n0 + rr) * LDF + m0 + 4 * g4 + j] = c[j];
    } else if (tid < 256 + NP) {
        const int i = tid - 256;
        float v = 0.f;
        for (int r = 0; r < NP; ++r) v = fmaf(sm.dT[r * LDF + i], sm.Mt[i * LDF + r], v);
        sm.dB[i] += v;
    }
    __syncthreads();
    // dA_rc = -sum_i M_ir W_ic (r > c), into TdA
    if (wave < 4) {
        const int m0 = 16 * (wave >> 1), n0 = 16 * (wave & 1);
        const f32x4 c = tile_mma<float, NP>(z, sm.Mt + m0 * LDF, LDF, sm.W + n0 * LDF, LDF, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = m0 + 4 * g4 + j, cc = n0 + rr;
            sm.TdA[r * LDF + cc] = r > cc ? -c[j] : 0.f;
        }
    }
    __syncthreads();
    hook2();
    // dbeta_r += sum_c dA_rc F_rc; dG from A: WA = dA o A, dG_r += sum_c WA_rc, dG_c -= sum_r WA_rc;
    // dKK_rc = dA_rc beta_r gamma_r/gamma_c, symmetrised into Wh
#pragma unroll 1
    for (int it = 0; it < 2; ++it) {
        const int r = 16 * it + 2 * wave + (lane >> 5), c = lane & 31;
        float bt = 0.f, wa = 0.f, sym = 0.f;
        if (r > c) {
            const float da = sm.TdA[r * LDF + c], e = ex(sm.G[r] - sm.G[c]);
            const float f = e * sm.KK[r * LDF + c];
            bt = da * f;
            wa = da * sm.bet[r] * f;
            sym = da * sm.bet[r] * e;
        } else if (c > r) {
            sym = sm.TdA[c * LDF + r] * sm.bet[c] * ex(sm.G[c] - sm.G[r]);
        }
        sm.Wh[r * LDM + c] = (_Float16)sym;
        const float wc = wa + __shfl_xor(wa, 32);
        const float br = half_total(bt, lane), wr = half_total(wa, lane);
        if (c == 0) {
            lds_add(&sm.dB[r], br);
            lds_add(&sm.part[wave][r], wr);
        }
        if (lane < 32 && wc != 0.f) lds_add(&sm.part[wave][c], -wc);
    }
    __syncthreads();
    // ---- dK = -Gamma dR S0^T + D Delta dS_n^T + [clean] (s E o Mc)^T Q + (dKK + dKK^T) K, with
    // the R-gate term dG_r -= gamma_r sum_a K_ra (dR S0^T)_ra
    {
        const f16x4 k0q = op_tr(sm.K, LDH, 0, c0, lane), k1q = op_tr(sm.K, LDH, 16, c0, lane);
        f16x4 q0q, q1q;
        if constexpr (CLEAN) {
            q0q = op_tr(sm.Q, LDH, 0, c0, lane);
            q1q = op_tr(sm.Q, LDH, 16, c0, lane);
        }
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            f32x4 c = tile_mma<_Float16, DD>(z, sm.dR + 16 * tm * LDH, LDH, sm.S0 + c0 * LDH, LDH, lane);
            const f32x4 d2 = tile_mma<_Float16, DD>(z, sm.Dl + 16 * tm * LDH, LDH, sm.dS + c0 * LDH, LDH, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, col = c0 + rr;
                rowg[tm][j] += c[j] * (float)sm.K[r * LDH + col];
                c[j] += ex(Gn - sm.G[r]) * d2[j];
            }
            if constexpr (CLEAN)
                c = mfma(op_tr(sm.dPh, LDM, 16, 16 * tm, lane), q1q, mfma(op_tr(sm.dPh, LDM, 0, 16 * tm, lane), q0q, c));
            c = mfma(op_row(sm.Wh, LDM, 16 * tm, 16, lane), k1q, mfma(op_row(sm.Wh, LDM, 16 * tm, 0, lane), k0q, c));
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, col = c0 + rr;
                if (r < nvalid) put_qk(add_qk, p.dk + (long)r * a.h_qk * DD + col, c[j] * inv);
            }
        }
    }
    {   // the row gate terms: this wave's partial sums
        const float dl = wave_total(dlast);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j;
                const float t = row_total(rowg[tm][j]);
                if (rr == 15) sm.part[wave][r] += r == NP - 1 ? t + dl : t;
            }
    }
    __syncthreads();
    if (wave == 0) {   // dg = reverse cumulative sum of dG (a 32-lane scan)
        float x = 0.f;
        if (lane < NP) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w) x += sm.part[w][lane];
        }
#pragma unroll
        for (int o = 1; o < NP; o <<= 1) {
            const float y = __shfl_down(x, o);
            if (lane + o < NP) x += y;
        }
        if (lane < nvalid) {
            p.dg[(long)lane * a.h_v] = x * inv;
            p.db[(long)lane * a.h_v] = sm.dB[lane] * inv;
        }
    }
    __syncthreads();
}

// The state after one block of nvalid positions (padded to 32) from the seed in S0 (LDS
// f16): S_n = gamma_n S0 + K^T D Delta, Delta = T (V - Gamma K S0), into out (fp32, the C-tile
// layout of a state: wave w holds column block w, row blocks 0 .. 7).  Stages K in K, V in R,
// M in Mh, Delta in Dl and the gates; S0's writer must have passed a barrier before the call's
// first one, and the call ends with a barrier, after which S0 may be rewritten.
__device__ __forceinline__ void block_fwd(Smem &sm, const StreamPtrs &p, const BwdArgs &a, int nvalid, float (&out)[8][4], int tid)
{
    const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15, c0 = 16 * wave;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    {
        const Row8<__bf16> k = load_rows(p.k, (long)a.h_qk * DD, nvalid, tid);
        const Row8<__bf16> v = load_rows(p.v, (long)a.h_v * DD, nvalid, tid);
        const bool ok = tid < NP && tid < nvalid;
        const float gx = ok ? p.g[(long)tid * a.h_v] : 0.f, bx = ok ? p.beta[(long)tid * a.h_v] : 0.f;
        store_rows(sm.K, k, tid);
        store_rows(sm.R, v, tid);
        if (tid < NP) {
            sm.bet[tid] = bx;
            sm.G[tid] = gx;
        }
    }
    __syncthreads();
    if (wave == 0) cum_gates(sm, lane);
    __syncthreads();
    const float Gn = sm.G[NP - 1], gn = ex(Gn);
    if (wave == 0) solve_m(sm, sm.K, lane);
    f16x4 s0q[8];
#pragma unroll
    for (int tm = 0; tm < 8; ++tm) s0q[tm] = op_tr(sm.S0, LDH, 16 * tm, c0, lane);
#pragma unroll
    for (int tm = 0; tm < 2; ++tm) {   // R = V - Gamma K S0
        f32x4 x = z;
#pragma unroll
        for (int kb = 0; kb < 8; ++kb) x = mfma(op_row(sm.K, LDH, 16 * tm, 16 * kb, lane), s0q[kb], x);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, c = c0 + rr;
            sm.R[r * LDH + c] = (_Float16)((float)sm.R[r * LDH + c] - sm.gam[r] * x[j]);
        }
    }
    __syncthreads();
    {   // Delta = T R (T_ri = M_ri beta_i)
        const f32x4 b0 = ld4(sm.bet + 4 * g4), b1 = ld4(sm.bet + 16 + 4 * g4);
        const f16x4 r0 = op_tr(sm.R, LDH, 0, c0, lane), r1 = op_tr(sm.R, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            const f16x4 t0 = scale4(op_row(sm.Mh, LDM, 16 * tm, 0, lane), b0);
            const f16x4 t1 = scale4(op_row(sm.Mh, LDM, 16 * tm, 16, lane), b1);
            const f32x4 d = mfma(t1, r1, mfma(t0, r0, z));
#pragma unroll
            for (int j = 0; j < 4; ++j) sm.Dl[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = (_Float16)d[j];
        }
    }
    __syncthreads();
    {   // S_n = gamma_n S0 + K^T (D o Delta), the B operands D o Delta scaled per position
        f32x4 d0, d1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            d0[e] = ex(Gn - sm.G[4 * g4 + e]);
            d1[e] = ex(Gn - sm.G[16 + 4 * g4 + e]);
        }
        const f16x4 b0 = scale4(op_tr(sm.Dl, LDH, 0, c0, lane), d0);
        const f16x4 b1 = scale4(op_tr(sm.Dl, LDH, 16, c0, lane), d1);
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            const f32x4 c =
                mfma(op_tr(sm.K, LDH, 16, 16 * tm, lane), b1, mfma(op_tr(sm.K, LDH, 0, 16 * tm, lane), b0, z));
#pragma unroll
            for (int j = 0; j < 4; ++j) out[tm][j] = gn * (float)s0q[tm][j] + c[j];
        }
    }
    __syncthreads();
}

namespace {

// Unit t of the (block, v-head) units ordered so that the r = h_v / h_qk v-heads of a q/k
// head (consecutive v-heads) are consecutive: t = ((gblk h_qk) + hq) r + i, v-head h = hq r + i.
// Each workgroup runs the units of a (block, q/k head) one after the other, so that its dq, dk
// rows are stored by the first (i = 0) and added to by the others: a fixed summation order,
// no atomics, nothing to clear.  Returns the unit's index in the per-(block, v-head) arrays.
__device__ __forceinline__ long unit_of(const BwdArgs &a, long t, long &gblk, int &h, int &hq, int &i)
{
    const int r = a.h_v / a.h_qk;
    const long gi = t / r;
    i = (int)(t % r);
    gblk = gi / a.h_qk;
    hq = (int)(gi % a.h_qk);
    h = hq * r + i;
    return gblk * a.h_v + h;
}

// The (sequence, first row, rows) of global block gblk: packed documents start on block
// boundaries, so a block lies inside one document.
__device__ __forceinline__ void block_unit(const BwdArgs &a, long gblk, int &n, long &p0, int &nvalid)
{
    if (a.seg) {
        // a segment's unit: the last sequence n with seg[n] <= gblk (one with no blocks in
        // the segment has seg[n] == seg[n + 1] and is passed over), block blk0 + gblk - seg[n]
        int lo = 0, hi = a.n_chains / a.h_v;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.seg[mid] <= gblk)
                lo = mid;
            else
                hi = mid;
        }
        n = lo;
        const long r0 = a.cu ? a.cu[n] : (long)n * a.T, r1 = a.cu ? a.cu[n + 1] : r0 + a.T;
        p0 = r0 + (a.blk0 + gblk - a.seg[n]) * a.L;
        const long rem = r1 - p0;
        nvalid = rem < 0 ? 0 : (rem < a.L ? (int)rem : a.L);
    } else if (a.cu) {
        p0 = gblk * a.L;
        int lo = 0, hi = a.n_docs;   // the last document with cu[d] <= p0
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.cu[mid] <= p0)
                lo = mid;
            else
                hi = mid;
        }
        n = lo;
        const long rem = a.cu[lo + 1] - p0;
        nvalid = (int)(rem < a.L ? rem : a.L);
    } else {
        n = (int)(gblk / a.nblk);
        const int b = (int)(gblk % a.nblk);
        p0 = (long)n * a.T + (long)b * a.L;
        const int rem = a.T - b * a.L;
        nvalid = rem < a.L ? rem : a.L;
    }
}

template <typename Od>
__device__ __forceinline__ StreamPtrs stream_ptrs(const BwdArgs &a, bool noisy, long p0, int h, int hq)
{
    const long qks = (long)a.h_qk * DD, vs = (long)a.h_v * DD;
    StreamPtrs p;
    p.q = static_cast<const __bf16 *>(noisy ? a.qn : a.q) + p0 * qks + hq * DD;
    p.k = static_cast<const __bf16 *>(noisy ? a.kn : a.k) + p0 * qks + hq * DD;
    p.v = static_cast<const __bf16 *>(noisy ? a.vn : a.v) + p0 * vs + h * DD;
    p.g = (noisy ? a.gn : a.g) + p0 * a.h_v + h;
    p.beta = (noisy ? a.betan : a.beta) + p0 * a.h_v + h;
    p.dout = static_cast<const Od *>(noisy ? a.doutn : a.dout) + p0 * vs + h * DD;
    p.dq = (noisy ? a.dqn : a.dq) + p0 * qks + hq * DD;
    p.dk = (noisy ? a.dkn : a.dk) + p0 * qks + hq * DD;
    p.dv = (noisy ? a.dvn : a.dv) + p0 * vs + h * DD;
    p.dg = (noisy ? a.dgn : a.dg) + p0 * a.h_v + h;
    p.db = (noisy ? a.dbn : a.db) + p0 * a.h_v + h;
    return p;
}

}  // namespace

// The part of a clean block's contribution to the state gradient at its start that does not
// depend on the gradient dh at its end.  With dDelta = s P^T dO + D K dh and dR = T^T dDelta,
//   dS0 = gamma_n dh + s Q^T Gamma dO - K^T Gamma T^T (s P^T dO) - K^T (U K) dh,  U = Gamma T^T D,
// so acc += s Q^T Gamma dO - K^T Gamma T^T (s P^T dO), and U K (32 x 128, U_ij = T_ji
// gamma_i gamma_n / gamma_j, upper triangular with |U_ij| <= |T_ji|) goes to uk and gamma_n to
// *gnb for the reverse scan.
// The clean rows are staged in R (q), dDl (k) and dO (do): the arrays block_bwd leaves dead
// after its dR / dQ phase, so that a persistent workgroup stages the next unit's rows there
// while it finishes the current one.  gx, bx: the gate and step size of position tid.
__device__ __forceinline__ void clean_prep(Smem &sm, const BwdArgs &a, float gx, float bx, float (&acc)[8][4], _Float16 *uk,
                           float *gnb, int tid)
{
    const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15, c0 = 16 * wave;
    const float s = a.scale;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    const _Float16 *Qs = sm.R, *Ks = sm.dDl;
    if (tid < NP) {
        sm.bet[tid] = bx;
        sm.G[tid] = gx;
    }
    __syncthreads();
    if (wave == 0) cum_gates(sm, lane);
    __syncthreads();
    const float Gn = sm.G[NP - 1];
    if (tid == 0) *gnb = ex(Gn);
    if (wave == 0) {   // M
        solve_m(sm, Ks, lane);
    } else if (wave >= 4) {   // P = (Q K^T) o Mc
        const int m0 = 16 * ((wave - 4) >> 1), n0 = 16 * ((wave - 4) & 1);
        const f32x4 qk = tile_mma<_Float16, DD>(z, Qs + m0 * LDH, LDH, Ks + n0 * LDH, LDH, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = m0 + 4 * g4 + j, i = n0 + rr;
            sm.Ph[r * LDM + i] = (_Float16)(i <= r ? qk[j] * ex(sm.G[r] - sm.G[i]) : 0.f);
        }
    }
    __syncthreads();
    {   // Y = s P^T dO -> Dl
        const f16x4 do0 = op_tr(sm.dO, LDH, 0, c0, lane), do1 = op_tr(sm.dO, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            const f32x4 c =
                mfma(op_tr(sm.Ph, LDM, 16, 16 * tm, lane), do1, mfma(op_tr(sm.Ph, LDM, 0, 16 * tm, lane), do0, z));
#pragma unroll
            for (int j = 0; j < 4; ++j) sm.Dl[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = (_Float16)(s * c[j]);
        }
    }
    for (int e = tid; e < NP * NP; e += 64 * kWaves) {   // U -> Wh
        const int i = e / NP, j = e % NP;
        sm.Wh[i * LDM + j] =
            (_Float16)(j >= i ? (float)sm.Mh[j * LDM + i] * sm.bet[i] * ex(sm.G[i] + Gn - sm.G[j]) : 0.f);
    }
    __syncthreads();
    // dR0 = T^T Y, as -Gamma dR0 in registers (B operands); acc += K^T (-Gamma dR0) + Q^T (s Gamma dO)
    f16x4 drq[2], sd[2];
    {
        const f16x4 y0 = op_tr(sm.Dl, LDH, 0, c0, lane), y1 = op_tr(sm.Dl, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            f16x4 t0, t1;
            tt_ops(sm, tm, lane, t0, t1);
            const f32x4 c = mfma(t1, y1, mfma(t0, y0, z));
            const f32x4 gm = ld4(sm.gam + 16 * tm + 4 * g4);
            drq[tm] = h4(-gm * c);
            // s Gamma dO: the transpose loads of dO scaled by s gamma of their rows
            sd[tm] = scale4(op_tr(sm.dO, LDH, 16 * tm, c0, lane), s * gm);
        }
    }
#pragma unroll
    for (int tm = 0; tm < 8; ++tm) {
        f32x4 c = mfma(op_tr(Ks, LDH, 0, 16 * tm, lane), drq[0], z);
        c = mfma(op_tr(Ks, LDH, 16, 16 * tm, lane), drq[1], c);
        c = mfma(op_tr(Qs, LDH, 0, 16 * tm, lane), sd[0], c);
        c = mfma(op_tr(Qs, LDH, 16, 16 * tm, lane), sd[1], c);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[tm][j] += c[j];
    }
    {   // U K -> uk
        const f16x4 k0q = op_tr(Ks, LDH, 0, c0, lane), k1q = op_tr(Ks, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            const f32x4 u = mfma(op_row(sm.Wh, LDM, 16 * tm, 16, lane), k1q, mfma(op_row(sm.Wh, LDM, 16 * tm, 0, lane), k0q, z));
#pragma unroll
            for (int j = 0; j < 4; ++j) uk[(16 * tm + 4 * g4 + j) * DD + c0 + rr] = (_Float16)u[j];
        }
    }
    __syncthreads();
}

// Phase 1: every noisy block: its gradients and its seed's gradient, plus (PREP) the
// dh-independent part of the clean block of the same position (clean_prep, run first: it
// needs no seed); both enter the state gradient at the block's start, whose sum is written
// to cterm (fp16, the precision of the dh it joins; per (block, v-head) 64 tiles of 16 x 16
// in row-major tile order, each tile stored lane-major in the MFMA result layout: lane
// 16 g + r holds rows 4 g .. 4 g + 3 of column r as one 8-byte vector, the layout both
// this kernel and the scan hold it in registers).  Without PREP (the further noisy views of
// the complementary-view backward, each seeded from the same clean state) the seed's
// gradient is added to cterm.  Persistent: one 160 KB workgroup per CU walks the units (global block,
// v-head) u = blockIdx.x, + gridDim.x, ...; the next unit's clean rows are loaded while the
// current unit finishes and staged into arrays it no longer uses, and each unit's seed and
// noisy rows are in flight while its clean prep runs.
template <typename Od, bool PREP>
__global__ void __launch_bounds__(512) bdgdn_bwd_noisy_kernel(BwdArgs a)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Smem &sm = *reinterpret_cast<Smem *>(smem_raw);
    // workgroup w takes the (block, q/k head) groups w, w + gridDim.x, ..., each as its r
    // consecutive units (unit_of)
    const int r = a.h_v / a.h_qk;
    long u = (long)blockIdx.x * r;
    auto next_unit = [&](long t) { return (t + 1) % r ? t + 1 : t + 1 + (long)(gridDim.x - 1) * r; };
    float cg = 0.f, cb = 0.f;   // the clean gate and step size of position tid of unit u
    if constexpr (PREP) {
        const int tid = threadIdx.x;
        int n, nvalid;
        long p0;
        long gb;
        int h, hq, vi;
        unit_of(a, u, gb, h, hq, vi);
        block_unit(a, gb, n, p0, nvalid);
        const BlockRows<Od, false> cin =
            load_block<Od, false>(stream_ptrs<Od>(a, false, p0, h, hq), a.h_qk, a.h_v, nvalid, tid);
        store_rows(sm.R, cin.q, tid);
        store_rows(sm.dDl, cin.k, tid);
        store_rows(sm.dO, cin.dout, tid, a.range[0]);
        cg = cin.g;
        cb = cin.b;
    }
    for (;;) {
        // the thread index made opaque per unit, so that the body's lane-dependent addresses
        // are recomputed rather than hoisted out of the loop (where they would stay live)
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15;
        const long un = next_unit(u);
        const bool more = un < a.n_units;
        int n, nvalid;
        long p0;
        long gb;
        int h, hq, vi;
        const long uw = unit_of(a, u, gb, h, hq, vi);   // the unit's workspace index
        block_unit(a, gb, n, p0, nvalid);
        const StreamPtrs pn = stream_ptrs<Od>(a, true, p0, h, hq);
        const SeedRegs seed = load_seed(a.seeds + (size_t)uw * DD * DD, tid);
        const BlockRows<Od, true> nin = load_block<Od, true>(pn, a.h_qk, a.h_v, nvalid, tid);
        float acc[8][4];
#pragma unroll
        for (int tm = 0; tm < 8; ++tm)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[tm][j] = 0.f;
        if constexpr (PREP) clean_prep(sm, a, cg, cb, acc, a.uk + uw * NP * DD, a.gnb + uw, tid);
        store_seed(sm.S0, seed, tid);   // made visible by block_bwd's first barrier
        BlockRows<Od, false> nxt;
        block_bwd<Mode::Noisy, Od>(
            sm, pn, a, nvalid, nin, acc, tid, vi > 0,
            [&] {
                if (PREP && more) {
                    int n2, nv2;
                    long q0;
                    long gb2;
                    int h2, hq2, vi2;
                    unit_of(a, un, gb2, h2, hq2, vi2);
                    block_unit(a, gb2, n2, q0, nv2);
                    nxt = load_block<Od, false>(stream_ptrs<Od>(a, false, q0, h2, hq2), a.h_qk, a.h_v, nv2, tid);
                }
            },
            [&] {
                if (PREP && more) {
                    store_rows(sm.R, nxt.q, tid);
                    store_rows(sm.dDl, nxt.k, tid);
                    store_rows(sm.dO, nxt.dout, tid, a.range[0]);
                    cg = nxt.g;
                    cb = nxt.b;
                }
            });
        f16x4 *dst = reinterpret_cast<f16x4 *>(a.cterm + (size_t)uw * DD * DD) + wave * 64 + lane;
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            f16x4 *p = dst + tm * 8 * 64;   // tile (tm, wave)
            f16x4 v;
            if constexpr (!PREP) v = *p;
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = (_Float16)(PREP ? acc[tm][j] : (float)v[j] + acc[tm][j]);
            *p = v;
        }
        if (!more) break;
        u = un;
    }
}

// Phase 1 for noisy blocks of two sub-blocks (blocks of 2 L positions, L = a.L <= 32, the
// clean stream cut into sub-blocks of L): one workgroup per (block, v-head).  The noisy block
// runs from the clean seed S0 of its first sub-block a through its two halves,
// S~1 = f_a(S0) and S~2 = f_b(S~1), and every position of both halves reads S~2, so that
//   dQ = s dO S~2^T (both halves' rows),  dS~2 = s (Q_a^T dO_a + Q_b^T dO_b);
// half b is then differentiated from S~1 with dS_n = dS~2 (Mode::Given: it has no outputs of
// its own), which gives its gradients and dS~1, and half a from S0 with dS_n = dS~1, which
// gives its gradients and the seed's gradient dS0.  With PREP, dS0 and the dh-independent
// term of clean sub-block a (clean_prep) are written together to cterm of a, and clean
// sub-block b's term to cterm of b; without PREP (a further view) dS0 is added to cterm of a.
template <typename Od, bool PREP>
__device__ __forceinline__ void pair_unit(Smem &sm, const BwdArgs &a, long t, int tid)
{
    const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15, c0 = 16 * wave;
    long m;   // the block of 2 L positions
    int h, hq, vi;
    unit_of(a, t, m, h, hq, vi);
    const bool add_qk = vi > 0;
    const int L2 = 2 * a.L;
    long p0, ga;   // its first row; the global index of its first sub-block
    int nv;        // its rows
    if (a.seg) {
        // a segment's noisy block: the last sequence n with segp[n] <= m, its noisy block
        // (blk0 / 2) + m - segp[n] (blk0 and the segment length are even)
        int lo = 0, hi = a.n_chains / a.h_v;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.segp[mid] <= m)
                lo = mid;
            else
                hi = mid;
        }
        const long lm = m - a.segp[lo];
        const long r0 = a.cu ? a.cu[lo] : (long)lo * a.T, r1 = a.cu ? a.cu[lo + 1] : r0 + a.T;
        p0 = r0 + (a.blk0 + 2 * lm) * a.L;
        const long rem = r1 - p0;
        nv = rem < 0 ? 0 : (rem < L2 ? (int)rem : L2);
        ga = a.seg[lo] + 2 * lm;
    } else if (a.cu) {
        p0 = m * L2;   // documents start on block boundaries
        int lo = 0, hi = a.n_docs;   // the last document with cu[d] <= p0
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.cu[mid] <= p0)
                lo = mid;
            else
                hi = mid;
        }
        const long rem = a.cu[lo + 1] - p0;
        nv = (int)(rem < L2 ? rem : L2);
        ga = p0 / a.L;
    } else {
        const long nb2 = (a.T + L2 - 1) / L2;
        const int n = (int)(m / nb2), b = (int)(m % nb2);
        p0 = (long)n * a.T + (long)b * L2;
        const int rem = a.T - b * L2;
        nv = rem < L2 ? rem : L2;
        ga = (long)n * a.nblk + 2 * b;
    }
    const int nva = nv < a.L ? nv : a.L, nvb = nv - nva;   // rows of the halves (nvb may be 0)
    const long ua = ga * a.h_v + h, ub = ua + a.h_v;
    const StreamPtrs pa = stream_ptrs<Od>(a, true, p0, h, hq), pb = stream_ptrs<Od>(a, true, p0 + a.L, h, hq);
    const long qks = (long)a.h_qk * DD, vs = (long)a.h_v * DD;
    const float s = a.scale, inv = a.range[1];
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    float st[8][4];   // a state in the C-tile layout
    // S~1 = f_a(S0) into S0; S~2 = f_b(S~1) into dS
    store_seed(sm.S0, load_seed(a.seeds + (size_t)ua * DD * DD, tid), tid);
    __syncthreads();
    block_fwd(sm, pa, a, nva, st, tid);
#pragma unroll
    for (int tm = 0; tm < 8; ++tm)
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.S0[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = (_Float16)st[tm][j];
    __syncthreads();
    asm volatile("" : "+v"(tid));   // lane-dependent addresses recomputed per phase, not kept live
    block_fwd(sm, pb, a, nvb, st, tid);
#pragma unroll
    for (int tm = 0; tm < 8; ++tm)
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.dS[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = (_Float16)st[tm][j];
    // the halves' q and do rows: Q_a in Q, dO_a in dO, Q_b in dR, dO_b in dDl
    store_rows(sm.Q, load_rows(pa.q, qks, nva, tid), tid);
    store_rows(sm.dO, load_rows(static_cast<const Od *>(pa.dout), vs, nva, tid), tid, a.range[0]);
    store_rows(sm.dR, load_rows(pb.q, qks, nvb, tid), tid);
    store_rows(sm.dDl, load_rows(static_cast<const Od *>(pb.dout), vs, nvb, tid), tid, a.range[0]);
    __syncthreads();
    // dQ = s dO S~2^T for the rows of both halves
#pragma unroll
    for (int x = 0; x < 2; ++x) {
        const _Float16 *dOx = x ? sm.dDl : sm.dO;
        const StreamPtrs &px = x ? pb : pa;
        const int nvx = x ? nvb : nva;
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
            const f32x4 c = tile_mma<_Float16, DD>(z, dOx + 16 * tm * LDH, LDH, sm.dS + c0 * LDH, LDH, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j;
                if (r < nvx) put_qk(add_qk, px.dq + (long)r * qks + c0 + rr, s * c[j] * inv);
            }
        }
    }
    // dS~2 = s (Q_a^T dO_a + Q_b^T dO_b), written over S~2 once every read of it is done
    f16x4 ds[8];
    {
        const f16x4 da0 = op_tr(sm.dO, LDH, 0, c0, lane), da1 = op_tr(sm.dO, LDH, 16, c0, lane);
        const f16x4 db0 = op_tr(sm.dDl, LDH, 0, c0, lane), db1 = op_tr(sm.dDl, LDH, 16, c0, lane);
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            f32x4 c = mfma(op_tr(sm.Q, LDH, 0, 16 * tm, lane), da0, z);
            c = mfma(op_tr(sm.Q, LDH, 16, 16 * tm, lane), da1, c);
            c = mfma(op_tr(sm.dR, LDH, 0, 16 * tm, lane), db0, c);
            c = mfma(op_tr(sm.dR, LDH, 16, 16 * tm, lane), db1, c);
            ds[tm] = h4(c * s);
        }
    }
    __syncthreads();
#pragma unroll
    for (int tm = 0; tm < 8; ++tm)
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.dS[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = ds[tm][j];
    // half b from S~1 (S0) with dS_n = dS~2 (dS): its gradients, and dS~1 into acc
    float acc[8][4];
#pragma unroll
    for (int tm = 0; tm < 8; ++tm)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[tm][j] = 0.f;
    asm volatile("" : "+v"(tid));
    block_bwd<Mode::Given, Od>(sm, pb, a, nvb, load_block<Od, true>(pb, a.h_qk, a.h_v, nvb, tid), acc, tid, add_qk, [] {},
                               [] {});
    // half a from the clean seed with dS_n = dS~1: its gradients, and dS0 into acc
#pragma unroll
    for (int tm = 0; tm < 8; ++tm)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            sm.dS[(16 * tm + 4 * g4 + j) * LDH + c0 + rr] = (_Float16)acc[tm][j];
            acc[tm][j] = 0.f;
        }
    store_seed(sm.S0, load_seed(a.seeds + (size_t)ua * DD * DD, tid), tid);
    asm volatile("" : "+v"(tid));
    block_bwd<Mode::Given, Od>(sm, pa, a, nva, load_block<Od, true>(pa, a.h_qk, a.h_v, nva, tid), acc, tid, add_qk, [] {},
                               [] {});
    if constexpr (PREP) {
        // clean sub-blocks a and b: their dh-independent terms (a's together with dS0)
#pragma unroll 1
        for (int x = 0; x < 2; ++x) {
            if (x == 1 && nvb <= 0) break;   // a partial last block without a second sub-block
            const long ux = x ? ub : ua;
            const int nvx = x ? nvb : nva;
            const BlockRows<Od, false> cin = load_block<Od, false>(stream_ptrs<Od>(a, false, p0 + x * a.L, h, hq),
                                                                   a.h_qk, a.h_v, nvx, tid);
            store_rows(sm.R, cin.q, tid);
            store_rows(sm.dDl, cin.k, tid);
            store_rows(sm.dO, cin.dout, tid, a.range[0]);
            if (x == 1) {
#pragma unroll
                for (int tm = 0; tm < 8; ++tm)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[tm][j] = 0.f;
            }
            clean_prep(sm, a, cin.g, cin.b, acc, a.uk + ux * NP * DD, a.gnb + ux, tid);
            f16x4 *dst = reinterpret_cast<f16x4 *>(a.cterm + (size_t)ux * DD * DD) + wave * 64 + lane;
#pragma unroll
            for (int tm = 0; tm < 8; ++tm) {
                f16x4 v;
#pragma unroll
                for (int j = 0; j < 4; ++j) v[j] = (_Float16)acc[tm][j];
                dst[tm * 8 * 64] = v;
            }
        }
    } else {
        f16x4 *dst = reinterpret_cast<f16x4 *>(a.cterm + (size_t)ua * DD * DD) + wave * 64 + lane;
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            f16x4 v = dst[tm * 8 * 64];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = (_Float16)((float)v[j] + acc[tm][j]);
            dst[tm * 8 * 64] = v;
        }
    }
}

// One workgroup per (block, q/k head): the pair units of its v-heads in turn.
template <typename Od, bool PREP>
__global__ void __launch_bounds__(512) bdgdn_bwd_pair_kernel(BwdArgs a)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Smem &sm = *reinterpret_cast<Smem *>(smem_raw);
    const int r = a.h_v / a.h_qk;
    for (int i = 0; i < r; ++i) {
        // the thread index made opaque per unit, so that lane-dependent addresses are
        // recomputed rather than hoisted out of the loop (where they would stay live)
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        pair_unit<Od, PREP>(sm, a, (long)blockIdx.x * r + i, tid);
    }
}

// Phase 3: every clean block, in parallel, from its seed and the gradient at its end (dh,
// written by the scan); one workgroup per (block, q/k head).
template <typename Od>
__global__ void __launch_bounds__(512) bdgdn_bwd_clean_kernel(BwdArgs a)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Smem &sm = *reinterpret_cast<Smem *>(smem_raw);
    const int r = a.h_v / a.h_qk;
    for (int i = 0; i < r; ++i) {   // the v-heads of this (block, q/k head) in turn
        int tid = threadIdx.x;       // opaque per unit, as in the noisy kernel
        asm volatile("" : "+v"(tid));
        long gblk;
        int h, hq, vi;
        unit_of(a, (long)blockIdx.x * r + i, gblk, h, hq, vi);
        int n, nvalid;
        long p0;
        block_unit(a, gblk, n, p0, nvalid);
        const size_t so = ((size_t)gblk * a.h_v + h) * DD * DD;
        const StreamPtrs pc = stream_ptrs<Od>(a, false, p0, h, hq);
        const SeedRegs seed = load_seed(a.seeds + so, tid);
        const SeedRegs dh = load_seed(a.dh + so, tid);   // fp16, tile-native
        const BlockRows<Od, true> in = load_block<Od, true>(pc, a.h_qk, a.h_v, nvalid, tid);
        store_seed(sm.S0, seed, tid);
        store_tiles(sm.dS, dh, tid);
        float no_acc[8][4] = {};   // the clean stream forms no dS0
        // its first barrier covers S0, dS; its last one the next v-head's stores
        block_bwd<Mode::Clean, Od>(sm, pc, a, nvalid, in, no_acc, tid, vi > 0, [] {}, [] {});
    }
}

// Phase 2: the reverse scan of the clean state gradient over the blocks of a (sequence,
// v-head) (a chain), one workgroup of NW waves per TC = 8 NW columns (the columns are
// independent):
//   dh_(b-1) = gamma_n dh_b + cterm_b - K^T Z,  Z = (U K) dh_b  (32 x TC),
// writing dh_b (the gradient at the end of block b; fp16, the precision phase 3 uses it in,
// tile-native) over cterm_b, which only this scan reads, for phase 3, and dh0 (fp32).  The operands of block b - 2 (U K, K, cterm, gamma_n) are
// loaded into registers while block b is computed.
namespace {
constexpr int LDK = NP + 8;   // f16 row stride of [*][32] tiles
constexpr int kScanWaves = 4;   // waves per workgroup (2: 16 columns, two workgroups per CU, was slower)
template <int TC> struct ScanSmem {
    _Float16 UK[NP * LDH];       // U K of the block (32 x 128)
    _Float16 dHt[TC * LDH];      // dh_b transposed: the tile's TC columns x 128 rows
    _Float16 Kr[2][NP * LDH];    // K (32 x 128, row-major; its transpose is read by transpose loads), two buffers
    _Float16 Zt[TC * LDK];       // Z transposed: TC columns x 32 positions
};
}  // namespace

template <int NW>
__global__ void __launch_bounds__(64 * NW) bdgdn_bwd_scan_kernel(BwdArgs a)
{
    constexpr int TC = 8 * NW;           // columns per workgroup
    constexpr int NT = DD / TC;          // column tiles per chain
    constexpr int RT = DD / (16 * NW);   // 16-row tiles of dh per wave
    constexpr int CT = TC / 16;          // 16-column tiles
    constexpr int NC = 8 / NW;           // 16-byte chunks of a 32 x 128 operand per thread
    __shared__ __align__(16) ScanSmem<TC> sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15;
    // the NT column tiles of a chain on one XCD (workgroups are dealt to the 8 XCDs in turn),
    // so that they read its U K and K rows through one L2
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int chain = (slot / NT) * 8 + xcd, v0 = TC * (slot % NT);
    if (chain >= a.n_chains) return;
    const int n = chain / a.h_v, h = chain % a.h_v, hq = h / (a.h_v / a.h_qk);
    long r0, r1;
    if (a.cu) {
        r0 = a.cu[n];
        r1 = a.cu[n + 1];
    } else {
        r0 = (long)n * a.T;
        r1 = r0 + a.T;
    }
    const int nb = (int)((r1 - r0 + a.L - 1) / a.L);
    // the blocks walked, blo .. bhi - 1, and the workspace unit of block b, gb0 + b: all the
    // chain's blocks by global index (documents start on block boundaries), or those of one
    // time segment numbered from seg[n]; the walk starts from dht where the chain ends in it,
    // else from the gradient the next segment left in carry, and ends in dh0 at the chain's
    // start, else in carry
    int blo = 0, bhi = nb;
    long gb0 = a.cu ? r0 / a.L : (long)n * a.nblk;
    bool from_dht = true, to_dh0 = true;
    if (a.seg) {
        blo = a.blk0;
        bhi = nb < a.blk0 + a.seg_len ? nb : a.blk0 + a.seg_len;
        // no blocks of this chain in the segment: nothing to do, but for an empty chain,
        // whose dh0 is dht, in the first segment
        if (bhi <= blo && !(nb == 0 && a.blk0 == 0)) return;
        gb0 = a.seg[n] - blo;
        from_dht = nb <= a.blk0 + a.seg_len;
        to_dh0 = a.blk0 == 0;
    }
    const size_t SS = (size_t)DD * DD;
    const long qks = (long)a.h_qk * DD;
    // dh tiles: wave w holds rows (128 / NW) w .. + 128 / NW - 1 (RT row tiles) of the TC columns
    const int rw = (DD / NW) * wave;
    float dh[RT][CT][4];
    const float *dht = a.dht ? a.dht + ((size_t)n * a.h_v + h) * SS : nullptr;
    float *carry = a.seg ? a.carry + ((size_t)n * a.h_v + h) * SS : nullptr;
    const float sg = a.range[0];
#pragma unroll
    for (int tl = 0; tl < RT; ++tl)
#pragma unroll
        for (int tn = 0; tn < CT; ++tn)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int e = (rw + 16 * tl + 4 * g4 + j) * DD + v0 + 16 * tn + rr;
                // the carry holds dh as the walk keeps it (times sigma)
                dh[tl][tn][j] = !from_dht ? carry[e] : (dht ? dht[e] * sg : 0.f);
            }
    // wait for these loads here, once: left pending into the loop, they would make every
    // step wait for all outstanding loads (the prefetch of the next blocks included)
#pragma unroll
    for (int tl = 0; tl < RT; ++tl)
#pragma unroll
        for (int tn = 0; tn < CT; ++tn)
#pragma unroll
            for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(dh[tl][tn][j]));
    // staging map of the 32 x 128 operands: NC consecutive 16-byte chunks of one row per thread
    const int sr = (tid * NC) >> 4, sc = ((tid * NC) & 15) * 8;
    // one block's operands in registers; three sets rotate so that the loads for blocks
    // b - 1 and b - 2 are in flight while block b is computed (no register copy waits on them)
    struct Ops {
        f16x8 uk[NC];
        bf16x8 k[NC];
        f16x4 cs[RT][CT];
        float gn;
    };
    auto fetch = [&](int b, Ops &o) {
        const long p0 = r0 + (long)b * a.L;
        const int nvalid = (int)(r1 - p0 < a.L ? r1 - p0 : a.L);
        const size_t unit = (size_t)(gb0 + b) * a.h_v + h;
        const f16x8 *u = reinterpret_cast<const f16x8 *>(a.uk + unit * NP * DD + sr * DD + sc);
#pragma unroll
        for (int i = 0; i < NC; ++i) o.uk[i] = u[i];
        if (sr < nvalid) {
            const bf16x8 *k = reinterpret_cast<const bf16x8 *>(static_cast<const __bf16 *>(a.k) + (p0 + sr) * qks +
                                                               hq * DD + sc);
#pragma unroll
            for (int i = 0; i < NC; ++i) o.k[i] = k[i];
        } else {
#pragma unroll
            for (int i = 0; i < NC; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j) o.k[i][j] = (__bf16)0.f;
        }
        // cterm tiles (rows rw / 16 + tl, columns v0 / 16 + tn), lane-major like the dh tiles
        const f16x4 *c = reinterpret_cast<const f16x4 *>(a.cterm + unit * SS) + lane;
#pragma unroll
        for (int tl = 0; tl < RT; ++tl)
#pragma unroll
            for (int tn = 0; tn < CT; ++tn) o.cs[tl][tn] = c[((rw / 16 + tl) * 8 + v0 / 16 + tn) * 64];
        // a vector load (the index made lane-opaque): a scalar load would be counted with the
        // LDS operations, and the wait before the next barrier would wait for it
        int z;
        asm volatile("v_mov_b32 %0, 0" : "=v"(z));
        o.gn = a.gnb[unit + z];
    };
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    auto step = [&](int b, const Ops &cur, Ops &nxt) {
        const int buf = b & 1;
        // dh_b goes to block b's cterm slot (tile-native, fp16), which this lane read two
        // steps earlier: the store is issued after that value's use below
        f16x4 *dhb = reinterpret_cast<f16x4 *>(a.dh + ((size_t)(gb0 + b) * a.h_v + h) * SS) + lane;
        f16x4 hv[RT][CT];
        // stage dh_b^T, U K, K^T of block b; every use of cur comes before the loads of block
        // b - 2 are issued, so that no wait for cur can also wait for those
#pragma unroll
        for (int tl = 0; tl < RT; ++tl)
#pragma unroll
            for (int tn = 0; tn < CT; ++tn) {
                const int r = rw + 16 * tl + 4 * g4, c = 16 * tn + rr;
                hv[tl][tn] = f16x4{(_Float16)dh[tl][tn][0], (_Float16)dh[tl][tn][1], (_Float16)dh[tl][tn][2],
                                   (_Float16)dh[tl][tn][3]};
                st4(sm.dHt + c * LDH + r, dh[tl][tn][0], dh[tl][tn][1], dh[tl][tn][2], dh[tl][tn][3]);
            }
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            *reinterpret_cast<f16x8 *>(sm.UK + sr * LDH + sc + 8 * i) = cur.uk[i];
            f16x8 kh;
#pragma unroll
            for (int j = 0; j < 8; ++j) kh[j] = (_Float16)(float)cur.k[i][j];
            *reinterpret_cast<f16x8 *>(sm.Kr[buf] + sr * LDH + sc + 8 * i) = kh;
        }
        // dh_b is in LDS now: keep gamma_n dh_b + cterm_b in its registers
#pragma unroll
        for (int tl = 0; tl < RT; ++tl)
#pragma unroll
            for (int tn = 0; tn < CT; ++tn)
#pragma unroll
                for (int j = 0; j < 4; ++j) dh[tl][tn][j] = cur.gn * dh[tl][tn][j] + (float)cur.cs[tl][tn][j];
#pragma unroll
        for (int tl = 0; tl < RT; ++tl)
#pragma unroll
            for (int tn = 0; tn < CT; ++tn) dhb[((rw / 16 + tl) * 8 + v0 / 16 + tn) * 64] = hv[tl][tn];
        if (b - 2 >= blo) fetch(b - 2, nxt);
        __syncthreads();
        {   // Z = (U K) dh_b: one 16 x 16 tile per wave (2 CT tiles over NW = 2 CT waves), stored transposed
            const int m0 = 16 * (wave / CT), n0 = 16 * (wave % CT);
            const f32x4 c = tile_mma<_Float16, DD>(z, sm.UK + m0 * LDH, LDH, sm.dHt + n0 * LDH, LDH, lane);
            st4(sm.Zt + (n0 + rr) * LDK + m0 + 4 * g4, c[0], c[1], c[2], c[3]);
        }
        __syncthreads();
#pragma unroll
        for (int tl = 0; tl < RT; ++tl)
#pragma unroll
            for (int tn = 0; tn < CT; ++tn) {
                // K^T Z: the A operand K^T by transpose loads of the row-major K, positions in two
                // 16-halves (the same k order as the Zt operand's)
                const int m0 = rw + 16 * tl;
                const f32x4 c = mfma(op_tr(sm.Kr[buf], LDH, 16, m0, lane), op_row(sm.Zt, LDK, 16 * tn, 16, lane),
                                     mfma(op_tr(sm.Kr[buf], LDH, 0, m0, lane), op_row(sm.Zt, LDK, 16 * tn, 0, lane), z));
#pragma unroll
                for (int j = 0; j < 4; ++j) dh[tl][tn][j] -= c[j];
            }
    };
    // three sets: block b's operands were loaded two steps earlier
    Ops o0, o1, o2;
    if (bhi - blo > 0) fetch(bhi - 1, o0);
    if (bhi - blo > 1) fetch(bhi - 2, o1);
    for (int b = bhi - 1; b >= blo; b -= 3) {
        step(b, o0, o2);
        if (b == blo) break;
        step(b - 1, o1, o0);
        if (b == blo + 1) break;
        step(b - 2, o2, o1);
    }
    float *d0 = !to_dh0 ? carry : (a.dh0 ? a.dh0 + ((size_t)n * a.h_v + h) * SS : nullptr);
    if (d0) {
        const float f = to_dh0 ? a.range[1] : 1.f;
#pragma unroll
        for (int tl = 0; tl < RT; ++tl)
#pragma unroll
            for (int tn = 0; tn < CT; ++tn)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    d0[(rw + 16 * tl + 4 * g4 + j) * DD + v0 + 16 * tn + rr] = dh[tl][tn][j] * f;
    }
}

// The range of the upstream gradients (dO, dO~ of every view, dht): each block's max |x| over
// its grid-stride share of every array into part[blockIdx.x].  With Od = bf16 the output
// gradients are bf16 (dht is always fp32).
__device__ __forceinline__ float absmax4(f32x4 v)
{
    return fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3])));
}
__device__ __forceinline__ float absmax8(bf16x8 v)
{
    float m = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf((float)v[j]));
    return m;
}
// max |x| over this block's contiguous segment of x[0 .. n), eight 16-byte loads in flight
// per thread
template <typename V, typename F>
__device__ __forceinline__ float range_max(const V *x, long n, float m, const F &absmax)
{
    const long seg = (n + gridDim.x - 1) / gridDim.x;
    const long end = min(n, seg * (blockIdx.x + 1));
    long e = seg * blockIdx.x + threadIdx.x;
    for (; e + 7 * 256 < end; e += 8 * 256) {
        V v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = x[e + u * 256];
#pragma unroll
        for (int u = 0; u < 8; ++u) m = fmaxf(m, absmax(v[u]));
    }
    for (; e < end; e += 256) m = fmaxf(m, absmax(x[e]));
    return m;
}
template <typename Od>
__global__ void __launch_bounds__(256) bdgdn_bwd_range_kernel(RangeArgs r)
{
    __shared__ float red[4];
    float m = 0.f;
    for (int i = 0; i < r.count; ++i) {
        const long n8 = r.n[i] / 8;   // 8-element vectors (every length is a multiple of 128)
        if (sizeof(Od) == 2 && !(i == r.count - 1 && r.last_f32))
            m = range_max(static_cast<const bf16x8 *>(r.arr[i]), n8, m, absmax8);
        else
            m = range_max(static_cast<const f32x4 *>(r.arr[i]), 2 * n8, m, absmax4);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) r.part[blockIdx.x] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// The blocks' maxima reduced to the power-of-two scale sigma that puts the largest upstream
// gradient in [4, 8), and its inverse: range[0] = sigma, range[1] = 1 / sigma (both 1 when
// every gradient is zero or one is not finite).  Every gradient is linear in the upstream
// gradients, so the block kernels work on sigma times them (fp16 operands keep their relative
// precision whatever the loss scale) and divide their fp32 results by sigma, exactly.
__global__ void __launch_bounds__(256) bdgdn_bwd_scale_kernel(const float *part, int n, float *range)
{
    __shared__ float red[4];
    float m = 0.f;
    bool bad = false;
    for (int i = threadIdx.x; i < n; i += 256) {
        const float v = part[i];
        bad |= !isfinite(v);
        m = fmaxf(m, v);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    const bool any_bad = __syncthreads_or(bad);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
        float sg = 1.f;
        if (!any_bad && m > 0.f) {
            int e;
            frexpf(m, &e);                       // m in [2^(e-1), 2^e)
            const int k = min(max(3 - e, -120), 120);
            sg = ldexpf(1.f, k);                 // sigma m in [4, 8)
        }
        range[0] = sg;
        range[1] = 1.f / sg;
    }
}

hipError_t launch_bwd_range(bool bf16_out, const RangeArgs &r, hipStream_t s)
{
    if (r.count < 1 || r.count > kRangeArrays) return hipErrorInvalidValue;
    if (bf16_out)
        hipLaunchKernelGGL(bdgdn_bwd_range_kernel<__bf16>, dim3(kRangeBlocks), dim3(256), 0, s, r);
    else
        hipLaunchKernelGGL(bdgdn_bwd_range_kernel<float>, dim3(kRangeBlocks), dim3(256), 0, s, r);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bdgdn_bwd_scale_kernel, dim3(1), dim3(256), 0, s, r.part, kRangeBlocks, r.range);
    return hipGetLastError();
}

size_t bwd_block_lds() { return sizeof(Smem); }

// The segment tables: thread k walks the sequences, counting the blocks of each inside
// segment k (and its noisy blocks of two sub-blocks, the last one possibly half).
__global__ void __launch_bounds__(64) bdgdn_bwd_seg_plan_kernel(const int32_t *cu, int n_seq, int T, int L,
                                                                int seg_len, int n_seg, int *seg, int *segp)
{
    const int k = blockIdx.x * 64 + threadIdx.x;
    if (k >= n_seg) return;
    int *o = seg + (long)k * (n_seq + 1), *op = segp + (long)k * (n_seq + 1);
    int acc = 0, accp = 0;
    for (int n = 0; n < n_seq; ++n) {
        o[n] = acc;
        op[n] = accp;
        const long len = cu ? (long)cu[n + 1] - cu[n] : T;
        const long nb = (len + L - 1) / L, rest = nb - (long)k * seg_len;
        const int cnt = rest <= 0 ? 0 : (rest < seg_len ? (int)rest : seg_len);
        acc += cnt;
        accp += (cnt + 1) / 2;
    }
    o[n_seq] = acc;
    op[n_seq] = accp;
}

hipError_t launch_bwd_seg_plan(const int32_t *cu, int n_seq, int T, int L, int seg_len, int n_seg, int *seg,
                               int *segp, hipStream_t s)
{
    if (n_seg <= 0 || n_seq <= 0 || L <= 0 || seg_len <= 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(bdgdn_bwd_seg_plan_kernel, dim3((n_seg + 63) / 64), dim3(64), 0, s, cu, n_seq, T, L, seg_len,
                       n_seg, seg, segp);
    return hipGetLastError();
}

hipError_t launch_bwd(bool bf16_out, const BwdArgs &a, const BwdView *more, int n_more, int n_chains,
                      long n_block_units, long n_pair_units, hipStream_t s)
{
    if (n_more < 0 || (n_more > 0 && !more)) return hipErrorInvalidValue;
    // one workgroup per (block, q/k head), running its r v-heads in turn (unit_of)
    const int r = a.h_v / a.h_qk;
    const long groups = n_block_units / r, pair_groups = n_pair_units / r;
    BwdArgs a2 = a;
    a2.n_units = n_block_units;
    // the noisy stream of a: its pointers replaced by those of view i
    auto with_view = [&](const BwdView &w) {
        BwdArgs b = a2;
        b.qn = w.q; b.kn = w.k; b.vn = w.v; b.gn = w.g; b.betan = w.beta; b.doutn = w.dout;
        b.dqn = w.dq; b.dkn = w.dk; b.dvn = w.dv; b.dgn = w.dg; b.dbn = w.db;
        return b;
    };
    // the persistent noisy kernels: one workgroup per CU (their LDS allows no more)
    int dev = 0, n_cu = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err == hipSuccess) err = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    const unsigned pgrid = (unsigned)(groups < n_cu ? groups : (n_cu > 0 ? n_cu : 1));
    auto run = [&](auto noisy, auto noisy_more, auto pair, auto pair_more, auto clean) {
        for (const void *f : {reinterpret_cast<const void *>(noisy), reinterpret_cast<const void *>(noisy_more),
                              reinterpret_cast<const void *>(pair), reinterpret_cast<const void *>(pair_more),
                              reinterpret_cast<const void *>(clean)}) {
            const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(Smem));
            if (e != hipSuccess) return e;
        }
        hipError_t e;
        if (pair_groups > 0) {   // noisy blocks of two sub-blocks
            hipLaunchKernelGGL(pair, dim3((unsigned)pair_groups), dim3(512), sizeof(Smem), s, a2);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            for (int i = 0; i < n_more; ++i) {   // in stream order: each adds its seed gradients
                hipLaunchKernelGGL(pair_more, dim3((unsigned)pair_groups), dim3(512), sizeof(Smem), s,
                                   with_view(more[i]));
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
        } else if (groups > 0) {
            hipLaunchKernelGGL(noisy, dim3(pgrid), dim3(512), sizeof(Smem), s, a2);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            for (int i = 0; i < n_more; ++i) {   // in stream order: each adds its seed gradients
                hipLaunchKernelGGL(noisy_more, dim3(pgrid), dim3(512), sizeof(Smem), s, with_view(more[i]));
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
        }
        constexpr int NT = DD / (8 * kScanWaves);   // column tiles per chain
        hipLaunchKernelGGL(bdgdn_bwd_scan_kernel<kScanWaves>, dim3((NT * n_chains + 8 * NT - 1) / (8 * NT) * 8 * NT),
                           dim3(64 * kScanWaves), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (groups > 0) {
            hipLaunchKernelGGL(clean, dim3((unsigned)groups), dim3(512), sizeof(Smem), s, a2);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        return hipSuccess;
    };
    return bf16_out ? run(bdgdn_bwd_noisy_kernel<__bf16, true>, bdgdn_bwd_noisy_kernel<__bf16, false>,
                          bdgdn_bwd_pair_kernel<__bf16, true>, bdgdn_bwd_pair_kernel<__bf16, false>,
                          bdgdn_bwd_clean_kernel<__bf16>)
                    : run(bdgdn_bwd_noisy_kernel<float, true>, bdgdn_bwd_noisy_kernel<float, false>,
                          bdgdn_bwd_pair_kernel<float, true>, bdgdn_bwd_pair_kernel<float, false>,
                          bdgdn_bwd_clean_kernel<float>);
}

}  // namespace bdgdn
