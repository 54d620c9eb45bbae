// ut.hpp -- the block-local UT transform of the Gated Delta Rule held in one wave's
// registers (Appendix "Chunk-corrected values", eq. f-blk): the cumulative gates of a
// block by a cross-lane scan, the Gram tiles of its keys on MFMA, and
// T = (I + A)^(-1) diag(beta) with
//     A_ri = beta_r 2^(G_r - G_i) (k_r . k_i)   (i < r),  G = cumulative log2-gates,
// for blocks of 16, 32 or 64 positions.  Shared by the one-kernel training forward, the
// serving kernels and the UT-transform kernel of the two-kernel schedule.
#pragma once

#include "common.hpp"

namespace bdgdn {

namespace ut {

typedef _Float16 E;
typedef f16x4 QE;

template <int CTRL> __device__ __forceinline__ float dpp(float v)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, true));
}
__device__ __forceinline__ float lane_value(float v, int l)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
// Inclusive prefix sum over lanes 0 .. 31: shifts by 1, 2, 4, 8 inside each 16-lane row,
// then the total of row 0 carried into row 1.
__device__ __forceinline__ float scan32(float x, int lane)
{
    x += dpp<0x111>(x);
    x += dpp<0x112>(x);
    x += dpp<0x114>(x);
    x += dpp<0x118>(x);
    const float r0 = lane_value(x, 15);
    return lane >= 16 && lane < 32 ? x + r0 : x;
}
__device__ __forceinline__ f32x4 mfma16(f16x4 a, f16x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 ld4f(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }

// Per-lane constants of the solve, element i of a 16 x 16 tile at row r = 4g + i,
// column n: the identity, the level-1 entries of A and A^T, and for the levels
// b = 2, 4, 8 an AND mask over the fp16 quad that keeps the entries of M_b^T (those above
// the diagonal whose row and column differ first in bit log2 b).
struct Consts {
    f32x4 one, m1lo, m1up;
    unsigned mk[3][2];
};
__device__ __forceinline__ void make_consts(Consts &u, int lane)
{
    const int g = lane >> 4, n = lane & 15;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = 4 * g + i, xr = r ^ n;
        u.one[i] = xr == 0 ? 1.f : 0.f;
        u.m1lo[i] = xr == 1 && r > n ? 1.f : 0.f;
        u.m1up[i] = xr == 1 && n > r ? 1.f : 0.f;
    }
#pragma unroll
    for (int l = 0; l < 3; ++l) {
        const int b = 2 << l;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            unsigned m = 0;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int r = 4 * g + 2 * h + e, xr = r ^ n;
                if (n > r && xr >= b && xr < 2 * b) m |= 0xffffu << (16 * e);
            }
            u.mk[l][h] = m;
        }
    }
}
__device__ __forceinline__ f16x4 and_mask(f16x4 q, const unsigned (&m)[2])
{
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    u32x2 w = __builtin_bit_cast(u32x2, q);
    w[0] &= m[0];
    w[1] &= m[1];
    return __builtin_bit_cast(f16x4, w);
}

// T = (I + A)^(-1) diag(beta) of one block of NB x 16 positions (NB = 1, 2 or 4), written
// row-major to LDS (T, row stride ts, fp16, every entry including the zeros above the
// diagonal), from the key-row quads kq[rb][kb] (lane (g, r): row 16 rb + r, columns
// 16 kb + 4g .. + 3) and the block's cumulative log2-gates Gs and step sizes Bs (LDS, one
// per position).
//
// Everything stays in registers.  With mfma16(q(X), q(Y)) = X^T Y for accumulator tiles
// X, Y (lane (g, n) holding rows 4g .. 4g + 3 of column n), a product needs its left
// factor as the accumulator of its transpose; so the solve carries each matrix together
// with its transpose.  (I + A)^(-1) is built by doubling the size of the inverted
// diagonal blocks: with D_b the inverse restricted to blocks of size b and M_b the part
// of A between the two b-halves of each 2b block,
//     D_2b = D_b - D_b M_b D_b,    D_2 = I - M_1,
// which is the block lower-triangular inverse formula, so no intermediate exceeds the
// entries of the inverse itself.  Inside a 16 x 16 tile the levels b = 1 .. 8 run on all
// diagonal tiles at once; the 16 -> 32 level joins pairs of tiles (X10 = -X11 A10 X00) and
// the 32 -> 64 level the two 32-blocks (X_hl = -X_hh A_hl X_ll, 2 x 2 tiles each).
// Products take fp16 operands and accumulate in fp32.  T is written from transposed tiles,
// so each lane writes four consecutive entries of a row.  Masked entries are selected, not
// branched on.  With log-gates g <= 0 the cumulative G is non-increasing, so every decay
// exponent kept (G_r - G_c, r >= c) is <= 0 and is evaluated as -|G_r - G_c|, which also
// keeps the discarded entries finite.  With BETA = false the inverse M = (I + A)^(-1) itself
// is written instead of T (the backward needs M where a step size is zero).  With BLKDIAG
// the positions form consecutive groups of nl (a power of two) with no coupling between
// groups: A_ri is kept only where r and i lie in the same group, so T is block diagonal
// (the transform of each group on its own).
template <int NB, int DKB, bool BETA = true, bool BLKDIAG = false>
__device__ __forceinline__ void solve_t(const QE (&kq)[NB][DKB], const float *Gs, const float *Bs, E *T, int ts,
                                        const Consts &us_, int lane, int nl = 0)
{
    static_assert(NB == 1 || NB == 2 || NB == 4, "blocks of 16, 32 or 64 positions");
    const int g = lane >> 4, n = lane & 15;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    // kk[bi][bj]: lane (g, n) = k_(16 bi + 4g + i) . k_(16 bj + n)   (bi <= bj only)
    f32x4 kk[NB][NB];
#pragma unroll
    for (int bi = 0; bi < NB; ++bi)
#pragma unroll
        for (int bj = bi; bj < NB; ++bj) {
            kk[bi][bj] = mma_q<E, DKB>(z, kq[bi], kq[bj]);
            if constexpr (BLKDIAG) {
                // positions r, i share a group of nl iff (r ^ i) < nl
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (((16 * bi + 4 * g + i) ^ (16 * bj + n)) >= nl) kk[bi][bj][i] = 0.f;
            }
        }
    // per-lane gates: rows 4g + i and column n of each 16-block
    f32x4 gr[NB], br[NB];
    float gc[NB], bc[NB];
#pragma unroll
    for (int rb = 0; rb < NB; ++rb) {
        gr[rb] = ld4f(Gs + 16 * rb + 4 * g);
        br[rb] = ld4f(Bs + 16 * rb + 4 * g);
        gc[rb] = Gs[16 * rb + n];
        bc[rb] = Bs[16 * rb + n];
    }
    // (A_(bj, bi))^T for bi < bj: lane (g, n) = A[16 bj + n][16 bi + 4g + i]
    auto a_t = [&](int bi, int bj) {
        f32x4 a;
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = bc[bj] * fexp2(-fabsf(gc[bj] - gr[bi][i])) * kk[bi][bj][i];
        return a;
    };
    // T tile (bi, bj) from the accumulator of its transpose X_(bi, bj)^T (times beta of the
    // columns)
    auto put = [&](int bi, int bj, f32x4 xt) {
        if constexpr (BETA)
            st_quad(T + (16 * bi + n) * ts + 16 * bj + 4 * g, quad_of<E>(xt * br[bj]));
        else
            st_quad(T + (16 * bi + n) * ts + 16 * bj + 4 * g, quad_of<E>(xt));
    };
    // diagonal tiles of A (below the diagonal) and A^T (above): one exponent serves both
    f32x4 D[NB], Dt[NB];
    f16x4 atq[NB];
#pragma unroll
    for (int t = 0; t < NB; ++t) {
        f32x4 at;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float e = fexp2(-fabsf(gr[t][i] - gc[t])) * kk[t][t][i];
            at[i] = bc[t] * e;
            D[t][i] = fmaf(-us_.m1lo[i], br[t][i] * e, us_.one[i]);
            Dt[t][i] = fmaf(-us_.m1up[i], at[i], us_.one[i]);
        }
        atq[t] = quad_of<E>(at);
    }
#pragma unroll
    for (int l = 0; l < 3; ++l)
#pragma unroll
        for (int t = 0; t < NB; ++t) {
            const f32x4 y = mfma16(and_mask(atq[t], us_.mk[l]), quad_of<E>(D[t]), z);   // M_b D_b
            const f16x4 ny = quad_of<E>(-y), dtq = quad_of<E>(Dt[t]);
            D[t] = mfma16(dtq, ny, D[t]);                                             // D_b - D_b M_b D_b
            Dt[t] = mfma16(ny, dtq, Dt[t]);                                           // and its transpose
        }
    // the diagonal tiles of T (their entries above the diagonal are exact zeros: every
    // product there has a zero factor)
#pragma unroll
    for (int t = 0; t < NB; ++t) put(t, t, Dt[t]);
    if constexpr (NB >= 2) {
        // 16 -> 32: per pair (2p, 2p + 1), Y = A10 X00, X10 = -X11 Y (and its transpose)
        f32x4 x10[NB / 2], x10t[NB / 2];
#pragma unroll
        for (int pr = 0; pr < NB / 2; ++pr) {
            const int lo = 2 * pr, hi = 2 * pr + 1;
            const f32x4 y = mfma16(quad_of<E>(a_t(lo, hi)), quad_of<E>(D[lo]), z);
            const f16x4 ny = quad_of<E>(-y);
            x10t[pr] = mfma16(ny, quad_of<E>(Dt[hi]), z);
            x10[pr] = mfma16(quad_of<E>(Dt[hi]), ny, z);
            put(hi, lo, x10t[pr]);
            st_quad(T + (16 * lo + n) * ts + 16 * hi + 4 * g, quad_of<E>(z));
        }
        if constexpr (NB == 4) {
            // 32 -> 64: Y = A_hl X_ll (tiles Y_bj,bl for bj in {2, 3}, bl in {0, 1}), then
            // X_hl = -X_hh Y, produced transposed
            const f16x4 a02 = quad_of<E>(a_t(0, 2)), a12 = quad_of<E>(a_t(1, 2));
            const f16x4 a03 = quad_of<E>(a_t(0, 3)), a13 = quad_of<E>(a_t(1, 3));
            const f16x4 d0 = quad_of<E>(D[0]), d1 = quad_of<E>(D[1]), x10q = quad_of<E>(x10[0]);
            const f16x4 ny20 = quad_of<E>(-mfma16(a12, x10q, mfma16(a02, d0, z)));   // -(A20 X00 + A21 X10)
            const f16x4 ny21 = quad_of<E>(-mfma16(a12, d1, z));                      // -A21 X11
            const f16x4 ny30 = quad_of<E>(-mfma16(a13, x10q, mfma16(a03, d0, z)));   // -(A30 X00 + A31 X10)
            const f16x4 ny31 = quad_of<E>(-mfma16(a13, d1, z));                      // -A31 X11
            const f16x4 dt2 = quad_of<E>(Dt[2]), dt3 = quad_of<E>(Dt[3]), x32t = quad_of<E>(x10t[1]);
            put(2, 0, mfma16(ny20, dt2, z));                                 // (X22 Y20)^T, negated
            put(2, 1, mfma16(ny21, dt2, z));
            put(3, 0, mfma16(ny30, dt3, mfma16(ny20, x32t, z)));             // (X32 Y20 + X33 Y30)^T
            put(3, 1, mfma16(ny31, dt3, mfma16(ny21, x32t, z)));
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int bj = 2; bj < 4; ++bj) st_quad(T + (16 * bi + n) * ts + 16 * bj + 4 * g, quad_of<E>(z));
        }
    }
}

}  // namespace ut

}  // namespace bdgdn
