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
// One workgroup per (sequence, v-head) walks its blocks in reverse with dh (fp32) in
// registers; the seed of every block comes from the split schedule's clean scan
// (launch_scan_states).  Products are 16x16x16 MFMA tiles on fp16 operands read from LDS
// through accessors (any transposition is an index swap), fp32 accumulation; the 32x32
// triangular solve and the n x n backward terms run in fp32.  Blocks are padded to 32
// positions with identity steps (k = 0, beta = 0, g = 0), which change nothing.
#include "common.hpp"
#include "kernels.hpp"

namespace bdgdn {

namespace {

constexpr int NP = 32;           // positions per (padded) block
constexpr int DD = 128;          // d_k = d_v
constexpr int LDH = DD + 8;      // f16 row stride of [*][128] LDS matrices
constexpr int LDF = NP + 1;      // fp32 row stride of [32][32] LDS matrices
constexpr int kWaves = 8;

struct Smem {
    _Float16 S0[DD * LDH];       // seed state (d_k x d_v)
    _Float16 dS[DD * LDH];       // dS_n operand (d_k x d_v)
    _Float16 Q[NP * LDH], K[NP * LDH], R[NP * LDH], dO[NP * LDH];
    _Float16 Dl[NP * LDH], dDl[NP * LDH], dR[NP * LDH];
    float KK[NP * LDF], P[NP * LDF], M[NP * LDF], E[NP * LDF], dT[NP * LDF], W[NP * LDF], dA[NP * LDF];
    float G[NP], gam[NP], bet[NP], dG[NP], dB[NP];
};

// acc += A(16 x K) B(K x 16) for the output tile whose first row is m0 and first column n0.
template <int KD, typename FA, typename FB>
__device__ __forceinline__ f32x4 mm_tile(f32x4 acc, int m0, int n0, const FA &fa, const FB &fb, int lane)
{
    const int r = lane & 15, kq = (lane >> 4) * 4;
#pragma unroll 1
    for (int k0 = 0; k0 < KD; k0 += 16) {
        f16x4 av, bv;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            av[j] = fa(m0 + r, k0 + kq + j);
            bv[j] = fb(k0 + kq + j, n0 + r);
        }
        acc = __builtin_amdgcn_mfma_f32_16x16x16f16(av, bv, acc, 0, 0, 0);
    }
    return acc;
}

__device__ __forceinline__ float ex(float x) { return __expf(x); }

// Workgroup sum of v added to *dst (LDS), from every thread.
__device__ __forceinline__ void lds_add(float *dst, float v) { atomicAdd(dst, v); }

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

template <typename In> __device__ __forceinline__ void stage_rows(_Float16 *dst, const In *src, long stride, int nvalid,
                                                                 int tid)
{
    // 32 rows x 128 values, 8 per thread
    const int r = tid >> 4, c = (tid & 15) * 8;
    _Float16 h[8];
    if (r < nvalid) {
        const In *p = src + (long)r * stride + c;
#pragma unroll
        for (int j = 0; j < 8; ++j) h[j] = (_Float16)to_f(p[j]);
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) h[j] = (_Float16)0.f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) dst[r * LDH + c + j] = h[j];
}

struct StreamPtrs {
    const __bf16 *q, *k, *v;   // first row of the block (q/k head hq, v head h)
    const float *g, *beta;     // first row (head h), stride h_v
    const void *dout;          // first row (head h)
    float *dq, *dk, *dv, *dg, *db;   // first row of the gradients
};

}  // namespace

// One block's backward.  For the clean stream dS (LDS, f16) and dsn (registers, fp32, the
// tile layout of the carried state gradient: wave w holds column block w, row blocks 0..7)
// hold dS_n on entry; for the noisy stream dS_n is formed here from the block-end readout
// (dsn is not read).  S0 (LDS f16) holds the seed.  Adds dS0 into acc (same layout).
template <bool CLEAN, typename Od>
__device__ void block_bwd(Smem &sm, const StreamPtrs &p, const BwdArgs &a, int nvalid, const float (&dsn)[8][4],
                          float (&acc)[8][4], int tid)
{
    const int lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15;
    const float s = a.scale;
    const long qks = (long)a.h_qk * DD, vs = (long)a.h_v * DD;
    // ---- stage rows and gates
    stage_rows(sm.Q, p.q, qks, nvalid, tid);
    stage_rows(sm.K, p.k, qks, nvalid, tid);
    stage_rows(sm.R, p.v, vs, nvalid, tid);   // V, becomes R below
    stage_rows(sm.dO, static_cast<const Od *>(p.dout), vs, nvalid, tid);
    if (tid < NP) {
        const bool ok = tid < nvalid;
        sm.bet[tid] = ok ? p.beta[(long)tid * a.h_v] : 0.f;
        sm.G[tid] = ok ? p.g[(long)tid * a.h_v] : 0.f;
        sm.dG[tid] = 0.f;
        sm.dB[tid] = 0.f;
    }
    __syncthreads();
    if (tid == 0) {   // local cumulative log-gates and their exponentials
        float c = 0.f;
        for (int i = 0; i < NP; ++i) {
            c += sm.G[i];
            sm.G[i] = c;
            sm.gam[i] = ex(c);
        }
    }
    __syncthreads();
    const float Gn = sm.G[NP - 1];
    const float gn = ex(Gn);
    auto hq = [](const _Float16 *m) { return [m](int r, int c) { return m[r * LDH + c]; }; };
    auto hqt = [](const _Float16 *m) { return [m](int r, int c) { return m[c * LDH + r]; }; };
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    // ---- KK = K K^T, P = (Q K^T) o Mc (clean); X = K S0 -> R = V - Gamma X; noisy dS_n = s Q^T dO
    if (wave < 4) {
        const int m0 = 16 * (wave >> 1), n0 = 16 * (wave & 1);
        f32x4 c = mm_tile<DD>(z, m0, n0, hq(sm.K), hqt(sm.K), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.KK[(m0 + 4 * g4 + j) * LDF + n0 + rr] = c[j];
        if constexpr (CLEAN) {
            c = mm_tile<DD>(z, m0, n0, hq(sm.Q), hqt(sm.K), lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = m0 + 4 * g4 + j, i = n0 + rr;
                sm.P[r * LDF + i] = i <= r ? c[j] * ex(sm.G[r] - sm.G[i]) : 0.f;
            }
        }
    }
#pragma unroll 1
    for (int tm = 0; tm < 2; ++tm) {   // X tiles: rows 16 tm, columns 16 wave
        const f32x4 x = mm_tile<DD>(z, 16 * tm, 16 * wave, hq(sm.K), hq(sm.S0), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, c = 16 * wave + rr;
            const float rv = (float)sm.R[r * LDH + c] - sm.gam[r] * x[j];
            sm.R[r * LDH + c] = (_Float16)rv;
        }
    }
    // dS_n (clean: given, fp32 in dsn; noisy: s Q^T dO, formed here in the dh tile layout):
    // its gamma_n dS_n share of dS0 and the gate term dG_last += gamma_n <dS_n, S0>
    {
        float wg = 0.f;
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            f32x4 c;
            if constexpr (CLEAN) {
#pragma unroll
                for (int j = 0; j < 4; ++j) c[j] = dsn[tm][j];
            } else {
                c = mm_tile<NP>(z, 16 * tm, 16 * wave, hqt(sm.Q), hq(sm.dO), lane) * s;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * tm + 4 * g4 + j, col = 16 * wave + rr;
                if constexpr (!CLEAN) sm.dS[r * LDH + col] = (_Float16)c[j];
                acc[tm][j] += gn * c[j];
                wg += c[j] * (float)sm.S0[r * LDH + col];
            }
        }
        wg = wave_sum(wg);
        if (lane == 0) lds_add(&sm.dG[NP - 1], gn * wg);
    }
    __syncthreads();
    // ---- A (fp32, into W), then M = (I + A)^-1 by forward substitution: one wave, lane c
    // computes column c of M in place (its own earlier entries are re-read from LDS)
    for (int e = tid; e < NP * NP; e += 64 * kWaves) {
        const int r = e / NP, i = e % NP;
        sm.W[r * LDF + i] = i < r ? sm.bet[r] * ex(sm.G[r] - sm.G[i]) * sm.KK[r * LDF + i] : 0.f;
    }
    __syncthreads();
    if (wave == 0 && lane < NP) {
        const int c = lane;
        for (int r = 0; r < NP; ++r) {
            float v = r == c ? 1.f : 0.f;
            for (int i = c; i < r; ++i) v = fmaf(-sm.W[r * LDF + i], sm.M[i * LDF + c], v);
            sm.M[r * LDF + c] = r < c ? 0.f : v;
        }
    }
    __syncthreads();
    // ---- Delta = T R, T_ri = M_ri beta_i
    auto Tacc = [&sm](int r, int i) { return (_Float16)(sm.M[r * LDF + i] * sm.bet[i]); };
#pragma unroll 1
    for (int tm = 0; tm < 2; ++tm) {
        const f32x4 c = mm_tile<NP>(z, 16 * tm, 16 * wave, Tacc, hq(sm.R), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.Dl[(16 * tm + 4 * g4 + j) * LDH + 16 * wave + rr] = (_Float16)c[j];
    }
    __syncthreads();
    // ---- E = dO Delta^T; dDelta = [clean] s P^T dO + D K dS_n, with the D-term gate gradient
    if (wave < 4) {
        const int m0 = 16 * (wave >> 1), n0 = 16 * (wave & 1);
        const f32x4 c = mm_tile<DD>(z, m0, n0, hq(sm.dO), hqt(sm.Dl), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.E[(m0 + 4 * g4 + j) * LDF + n0 + rr] = c[j];
    }
#pragma unroll 1
    for (int tm = 0; tm < 2; ++tm) {
        const f32x4 kds = mm_tile<DD>(z, 16 * tm, 16 * wave, hq(sm.K), hq(sm.dS), lane);
        f32x4 pd = z;
        if constexpr (CLEAN) {
            auto Pt = [&sm](int r, int i) { return (_Float16)sm.P[i * LDF + r]; };
            pd = mm_tile<NP>(z, 16 * tm, 16 * wave, Pt, hq(sm.dO), lane);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, c = 16 * wave + rr;
            const float Dr = ex(Gn - sm.G[r]);
            sm.dDl[r * LDH + c] = (_Float16)(s * pd[j] + Dr * kds[j]);
            // D-term of the gates: w_r = D_r sum_j (K dS_n)_rj Delta_rj -> dG_last += w, dG_r -= w
            float w = Dr * kds[j] * (float)sm.Dl[r * LDH + c];
            w += __shfl_xor(w, 1);
            w += __shfl_xor(w, 2);
            w += __shfl_xor(w, 4);
            w += __shfl_xor(w, 8);
            if (rr == 0) {
                lds_add(&sm.dG[r], -w);
                lds_add(&sm.dG[NP - 1], w);
            }
        }
    }
    __syncthreads();
    // ---- dR = T^T dDelta (= dV); dQ
    auto Tt = [&sm](int i, int r) { return (_Float16)(sm.M[r * LDF + i] * sm.bet[i]); };
#pragma unroll 1
    for (int tm = 0; tm < 2; ++tm) {
        const f32x4 c = mm_tile<NP>(z, 16 * tm, 16 * wave, Tt, hq(sm.dDl), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, col = 16 * wave + rr;
            sm.dR[r * LDH + col] = (_Float16)c[j];
            if (r < nvalid) p.dv[(long)r * a.h_v * DD + col] = c[j];
        }
    }
    // dQ = [clean] s Gamma (dO S0^T) + (s E o Mc) K;  [noisy] s gamma_n (dO S0^T) + s (E D) K
    auto dPm = [&sm, s, Gn](int r, int i) {
        if constexpr (CLEAN) return (_Float16)(i <= r ? s * sm.E[r * LDF + i] * ex(sm.G[r] - sm.G[i]) : 0.f);
        else return (_Float16)(s * sm.E[r * LDF + i] * ex(Gn - sm.G[i]));
    };
#pragma unroll 1
    for (int tm = 0; tm < 2; ++tm) {
        f32x4 c = mm_tile<DD>(z, 16 * tm, 16 * wave, hq(sm.dO), hqt(sm.S0), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, col = 16 * wave + rr;
            if constexpr (CLEAN) {
                // gate term of Gamma Q S0: dG_r += s gamma_r sum_a Q_ra (dO S0^T)_ra
                float w = s * sm.gam[r] * c[j] * (float)sm.Q[r * LDH + col];
                w += __shfl_xor(w, 1);
                w += __shfl_xor(w, 2);
                w += __shfl_xor(w, 4);
                w += __shfl_xor(w, 8);
                if (rr == 0) lds_add(&sm.dG[r], w);
                c[j] *= s * sm.gam[r];
            } else {
                c[j] *= s * gn;
            }
        }
        c = mm_tile<NP>(c, 16 * tm, 16 * wave, dPm, hq(sm.K), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, col = 16 * wave + rr;
            if (r < nvalid) {
                float *dst = p.dq + (long)r * a.h_qk * DD + col;
                if (a.atomic_qk)
                    atomicAdd(dst, c[j]);
                else
                    *dst = c[j];
            }
        }
    }
    // clean: gates of Mc, W = s E o P: dG_r += sum_i W_ri, dG_i -= sum_r W_ri
    if constexpr (CLEAN) {
        for (int e = tid; e < NP * NP; e += 64 * kWaves) {
            const int r = e / NP, i = e % NP;
            const float w = s * sm.E[r * LDF + i] * sm.P[r * LDF + i];
            if (w != 0.f) {
                lds_add(&sm.dG[r], w);
                lds_add(&sm.dG[i], -w);
            }
        }
    }
    __syncthreads();
    // ---- dT = dDelta R^T; dS0 into acc
    if (wave < 4) {
        const int m0 = 16 * (wave >> 1), n0 = 16 * (wave & 1);
        const f32x4 c = mm_tile<DD>(z, m0, n0, hq(sm.dDl), hqt(sm.R), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) sm.dT[(m0 + 4 * g4 + j) * LDF + n0 + rr] = c[j];
    }
    // dS0 += [clean] s Q^T Gamma dO - K^T Gamma dR (gamma_n dS_n was added above)
    {
        auto sgdo = [&sm, s](int i, int c) { return (_Float16)(s * sm.gam[i] * (float)sm.dO[i * LDH + c]); };
        auto mgdr = [&sm](int i, int c) { return (_Float16)(-sm.gam[i] * (float)sm.dR[i * LDH + c]); };
#pragma unroll
        for (int tm = 0; tm < 8; ++tm) {
            f32x4 c = mm_tile<NP>(z, 16 * tm, 16 * wave, hqt(sm.K), mgdr, lane);
            if constexpr (CLEAN) c = mm_tile<NP>(c, 16 * tm, 16 * wave, hqt(sm.Q), sgdo, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[tm][j] += c[j];
        }
    }
    __syncthreads();
    // ---- dbeta, dA = strictly lower part of -M^T (dT diag beta) M^T (fp32)
    // W = dT diag(beta) M^T  (W_rc = sum_i dT_ri beta_i M_ci)
    for (int e = tid; e < NP * NP; e += 64 * kWaves) {
        const int r = e / NP, c = e % NP;
        float v = 0.f;
        for (int i = 0; i < NP; ++i) v = fmaf(sm.dT[r * LDF + i] * sm.bet[i], sm.M[c * LDF + i], v);
        sm.W[r * LDF + c] = v;
    }
    if (tid < NP) {   // dbeta_i += sum_r dT_ri M_ri
        float v = 0.f;
        for (int r = 0; r < NP; ++r) v = fmaf(sm.dT[r * LDF + tid], sm.M[r * LDF + tid], v);
        sm.dB[tid] += v;
    }
    __syncthreads();
    // dA_rc = -sum_i M_ir W_ic (r > c)
    for (int e = tid; e < NP * NP; e += 64 * kWaves) {
        const int r = e / NP, c = e % NP;
        float v = 0.f;
        if (r > c)
            for (int i = 0; i < NP; ++i) v = fmaf(-sm.M[i * LDF + r], sm.W[i * LDF + c], v);
        sm.dA[r * LDF + c] = v;
    }
    __syncthreads();
    // dbeta_r += sum_c dA_rc F_rc; dG from A: WA = dA o A, dG_r += sum_c WA_rc, dG_c -= sum_r WA_rc;
    // dKK_rc = dA_rc beta_r gamma_r/gamma_c, symmetrised into W
    for (int e = tid; e < NP * NP; e += 64 * kWaves) {
        const int r = e / NP, c = e % NP;
        const float da = sm.dA[r * LDF + c];
        float sym = 0.f;
        if (r > c) {
            const float f = ex(sm.G[r] - sm.G[c]) * sm.KK[r * LDF + c];
            lds_add(&sm.dB[r], da * f);
            const float wa = da * sm.bet[r] * f;
            if (wa != 0.f) {
                lds_add(&sm.dG[r], wa);
                lds_add(&sm.dG[c], -wa);
            }
            sym = da * sm.bet[r] * ex(sm.G[r] - sm.G[c]);
        } else if (c > r) {
            sym = sm.dA[c * LDF + r] * sm.bet[c] * ex(sm.G[c] - sm.G[r]);
        }
        sm.W[r * LDF + c] = sym;
    }
    __syncthreads();
    // ---- dK = - Gamma dR S0^T + D Delta dS_n^T + [clean] (s E o Mc)^T Q + (dKK + dKK^T) K, with
    // the R-gate term dG_r -= gamma_r sum_a K_ra (dR S0^T)_ra; then dg, dbeta
    auto Wacc = [&sm](int r, int c) { return (_Float16)sm.W[r * LDF + c]; };
#pragma unroll 1
    for (int tm = 0; tm < 2; ++tm) {
        f32x4 c = mm_tile<DD>(z, 16 * tm, 16 * wave, hq(sm.dR), hqt(sm.S0), lane);
        const f32x4 d2 = mm_tile<DD>(z, 16 * tm, 16 * wave, hq(sm.Dl), hqt(sm.dS), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, col = 16 * wave + rr;
            float w = sm.gam[r] * c[j] * (float)sm.K[r * LDH + col];
            w += __shfl_xor(w, 1);
            w += __shfl_xor(w, 2);
            w += __shfl_xor(w, 4);
            w += __shfl_xor(w, 8);
            if (rr == 0) lds_add(&sm.dG[r], -w);
            c[j] = -sm.gam[r] * c[j] + ex(Gn - sm.G[r]) * d2[j];
        }
        if constexpr (CLEAN) {
            auto dPmT = [&sm, s](int i, int r) {
                return (_Float16)(i <= r ? s * sm.E[r * LDF + i] * ex(sm.G[r] - sm.G[i]) : 0.f);
            };
            c = mm_tile<NP>(c, 16 * tm, 16 * wave, dPmT, hq(sm.Q), lane);
        }
        c = mm_tile<NP>(c, 16 * tm, 16 * wave, Wacc, hq(sm.K), lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * tm + 4 * g4 + j, col = 16 * wave + rr;
            if (r < nvalid) {
                float *dst = p.dk + (long)r * a.h_qk * DD + col;
                if (a.atomic_qk)
                    atomicAdd(dst, c[j]);
                else
                    *dst = c[j];
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        float c = 0.f;
        for (int i = NP - 1; i >= 0; --i) {
            c += sm.dG[i];
            if (i < nvalid) {
                p.dg[(long)i * a.h_v] = c;
                p.db[(long)i * a.h_v] = sm.dB[i];
            }
        }
    }
    __syncthreads();
}

template <typename Od>
__global__ void __launch_bounds__(512) bdgdn_bwd_chain_kernel(BwdArgs a)
{
    extern __shared__ __align__(16) unsigned char smem_raw[];
    Smem &sm = *reinterpret_cast<Smem *>(smem_raw);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g4 = lane >> 4, rr = lane & 15;
    const int n = blockIdx.x / a.h_v, h = blockIdx.x % a.h_v;
    const int hq = h / (a.h_v / a.h_qk);
    long r0, r1;
    if (a.cu) {
        r0 = a.cu[n];
        r1 = a.cu[n + 1];
    } else {
        r0 = (long)n * a.T;
        r1 = r0 + a.T;
    }
    const int nb = (int)((r1 - r0 + a.L - 1) / a.L);
    const size_t SS = (size_t)DD * DD;
    float dh[8][4], acc[8][4];
    const float *dht = a.dht ? a.dht + ((size_t)n * a.h_v + h) * SS : nullptr;
#pragma unroll
    for (int tm = 0; tm < 8; ++tm)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            dh[tm][j] = dht ? dht[(16 * tm + 4 * g4 + j) * DD + 16 * wave + rr] : 0.f;
    const long qks = (long)a.h_qk * DD, vs = (long)a.h_v * DD;
    for (int b = nb - 1; b >= 0; --b) {
        const long p0 = r0 + (long)b * a.L;
        const int nvalid = (int)(r1 - p0 < a.L ? r1 - p0 : a.L);
        const long gblk = a.cu ? p0 / a.L : (long)n * a.nblk + b;
        const float *seed = a.seeds + ((size_t)gblk * a.h_v + h) * SS;
        // seed (f16) and dS_n = dh (f16 operand copy; fp32 in registers)
        for (int e = tid * 4; e < DD * DD; e += 512 * 4) {
            const f32x4 v = *reinterpret_cast<const f32x4 *>(seed + e);
            const int r = e / DD, c = e % DD;
#pragma unroll
            for (int j = 0; j < 4; ++j) sm.S0[r * LDH + c + j] = (_Float16)v[j];
        }
#pragma unroll
        for (int tm = 0; tm < 8; ++tm)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                sm.dS[(16 * tm + 4 * g4 + j) * LDH + 16 * wave + rr] = (_Float16)dh[tm][j];
                acc[tm][j] = 0.f;
            }
        __syncthreads();
        StreamPtrs pc, pn;
        pc.q = static_cast<const __bf16 *>(a.q) + (p0 * a.h_qk + hq) * DD;
        pc.k = static_cast<const __bf16 *>(a.k) + (p0 * a.h_qk + hq) * DD;
        pc.v = static_cast<const __bf16 *>(a.v) + (p0 * a.h_v + h) * DD;
        pc.g = a.g + p0 * a.h_v + h;
        pc.beta = a.beta + p0 * a.h_v + h;
        pc.dout = static_cast<const Od *>(a.dout) + p0 * vs + h * DD;
        pc.dq = a.dq + p0 * qks + hq * DD;
        pc.dk = a.dk + p0 * qks + hq * DD;
        pc.dv = a.dv + p0 * vs + h * DD;
        pc.dg = a.dg + p0 * a.h_v + h;
        pc.db = a.db + p0 * a.h_v + h;
        pn.q = static_cast<const __bf16 *>(a.qn) + (p0 * a.h_qk + hq) * DD;
        pn.k = static_cast<const __bf16 *>(a.kn) + (p0 * a.h_qk + hq) * DD;
        pn.v = static_cast<const __bf16 *>(a.vn) + (p0 * a.h_v + h) * DD;
        pn.g = a.gn + p0 * a.h_v + h;
        pn.beta = a.betan + p0 * a.h_v + h;
        pn.dout = static_cast<const Od *>(a.doutn) + p0 * vs + h * DD;
        pn.dq = a.dqn + p0 * qks + hq * DD;
        pn.dk = a.dkn + p0 * qks + hq * DD;
        pn.dv = a.dvn + p0 * vs + h * DD;
        pn.dg = a.dgn + p0 * a.h_v + h;
        pn.db = a.dbn + p0 * a.h_v + h;
        block_bwd<true, Od>(sm, pc, a, nvalid, dh, acc, tid);
        block_bwd<false, Od>(sm, pn, a, nvalid, dh, acc, tid);
#pragma unroll
        for (int tm = 0; tm < 8; ++tm)
#pragma unroll
            for (int j = 0; j < 4; ++j) dh[tm][j] = acc[tm][j];
    }
    if (a.dh0) {
        float *d0 = a.dh0 + ((size_t)n * a.h_v + h) * SS;
#pragma unroll
        for (int tm = 0; tm < 8; ++tm)
#pragma unroll
            for (int j = 0; j < 4; ++j) d0[(16 * tm + 4 * g4 + j) * DD + 16 * wave + rr] = dh[tm][j];
    }
}

__global__ void __launch_bounds__(256) bdgdn_bwd_zero_kernel(float *p, long n)
{
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) p[i] = 0.f;
}

size_t bwd_chain_lds() { return sizeof(Smem); }

hipError_t launch_bwd(bool bf16_out, const BwdArgs &a, int n_units, long qk_elems, hipStream_t s)
{
    if (a.atomic_qk) {
        for (float *p : {a.dq, a.dk, a.dqn, a.dkn}) {
            hipLaunchKernelGGL(bdgdn_bwd_zero_kernel, dim3(1024), dim3(256), 0, s, p, qk_elems);
            const hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    auto run = [&](auto kern) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)sizeof(Smem));
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, dim3(n_units), dim3(512), sizeof(Smem), s, a);
        return hipGetLastError();
    };
    return bf16_out ? run(bdgdn_bwd_chain_kernel<__bf16>) : run(bdgdn_bwd_chain_kernel<float>);
}

}  // namespace bdgdn
