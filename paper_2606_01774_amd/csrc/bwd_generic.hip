// bwd_generic.hip -- the per-step backward of the two-stream training forward (Appendix
// "Backward primitives": eq. per-step-bwd for each step, the noisy block-end readout
// backward eq. noisy-readout-bwd, and the block-level chain rule eq. dh-block-recursion),
// in fp32, for the shapes outside the block-form backward of bwd_kernels.hip: fp32 inputs,
// d_k or d_v of 64, blocks of 33 to 64 positions.
//
// Forward step t (column by column of the d_k x d_v state, alpha = exp g):
//     u = v - alpha S^T k,   S' = alpha S + beta k u^T,   clean o = s S'^T q.
// Its backward, from the gradient dS' of S':
//     w = dS'^T k,  dv = beta w,  dbeta = w . u,  dk = beta (dS' u - alpha S w),
//     dS^ = dS' - beta k w^T,  dg = <dS^, alpha S>,  dS = alpha dS^,
// and a clean step first adds s q do^T to dS' and gives dq = s S' do.  A noisy block is
// seeded with the clean state at its start and every position reads its end state S~:
// dS~ = s sum_l q_l do_l^T and dq_l = s S~ do_l; the gradient of its seed joins the clean
// state gradient at the block's start.
//
// One wave per (sequence or document, v-head, 16-column tile of d_v): lane (rg, c) holds
// column c of the tile, rows rg * d_k/4 .. rg * d_k/4 + d_k/4 - 1.  The wave walks the blocks
// backwards.  The clean states at every eighth block start come from a forward pass (the
// checkpoint kernel); a group of eight blocks is re-run forward into a per-wave scratch of
// block-start states, and inside a block the states before every eighth position are kept in
// LDS and each span of eight positions is recomputed before its backward steps.  Gradients
// summed over columns (dq, dk, dg, dbeta) are added with fp32 atomics (summation order not
// fixed); dv and dh0 are written once.
#include "bwd.hpp"
#include "common.hpp"
#include "kernels.hpp"

namespace bdgdn {

namespace {

constexpr int kStride = 8;   // blocks per checkpoint group
constexpr int kSpan = 8;     // positions per recomputed span
constexpr int kMaxSpans = 8; // blocks of up to 64 positions

template <int NR, typename In>
__device__ __forceinline__ void load_row(float (&x)[NR], const In *p)
{
    if constexpr (sizeof(In) == 2) {
#pragma unroll
        for (int u = 0; u < NR / 8; ++u) {
            const bf16x8 b = *reinterpret_cast<const bf16x8 *>(p + 8 * u);
#pragma unroll
            for (int e = 0; e < 8; ++e) x[8 * u + e] = (float)b[e];
        }
    } else {
#pragma unroll
        for (int u = 0; u < NR / 4; ++u) {
            const f32x4 b = *reinterpret_cast<const f32x4 *>(p + 4 * u);
#pragma unroll
            for (int e = 0; e < 4; ++e) x[4 * u + e] = b[e];
        }
    }
}
template <typename T> __device__ __forceinline__ float ld1(const T *p) { return to_f(*p); }

__device__ __forceinline__ float xor_sum(float x, int m) { return x + __shfl_xor(x, m, 64); }
// sum over the four row groups of a column (lanes c, c + 16, c + 32, c + 48)
__device__ __forceinline__ float col_sum(float x) { return xor_sum(xor_sum(x, 16), 32); }
__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) x = xor_sum(x, m);
    return x;
}

// Sum of x over the 16 column lanes of a row group, for every row: a butterfly that halves
// the rows each lane keeps; lane (rg, c) ends with the NR / 16 row sums starting at *row0.
template <int NR>
__device__ __forceinline__ void row_sums(float (&x)[NR], int c, int &row0)
{
    int base = 0;
#pragma unroll
    for (int b = 8, n = NR; b >= 1; b >>= 1) {
        n >>= 1;
        const bool up = (c & b) != 0;
#pragma unroll
        for (int j = 0; j < n; ++j) {
            const float send = up ? x[j] : x[n + j];
            const float keep = up ? x[n + j] : x[j];
            x[j] = keep + __shfl_xor(send, b, 64);
        }
        if (up) base += n;
    }
    row0 = base;
}

struct GenStream {
    const void *q, *k, *v;
    const float *g, *beta;
    const void *dout;
    float *dq, *dk, *dv, *dg, *db;
};
constexpr int kGenStreams = 5;   // the clean stream and up to four noisy views

struct GenArgs {
    GenStream st[kGenStreams];   // 0 clean, 1 .. n_views noisy
    int n_views;
    const int32_t *cu;           // packed documents, or null
    int n_seq;
    const float *h0, *dht;
    float *dh0;
    float *ckpt;                 // clean state before every kStride-th block of every chain
    float *scratch;              // per wave: the block-start states of its current group
    int T, L, h_qk, h_v, dk, dv, n_tiles;
    float scale;
    int ck_off[kMaxOrder + 1];   // packed: checkpoint groups of the documents before each one
};

template <typename In, typename Out, int DK>
struct Gen {
    static constexpr int NR = DK / 4;             // rows per lane
    static constexpr int ST = NR * 64;            // floats of one tile state in LDS
    static constexpr int BYTES = (kMaxSpans + kSpan) * ST * 4 + kSpan * 64 * 4;

    const GenArgs &a;
    int lane, c, rg;
    int seq, h, hq, tile;
    long base, len;
    int nb;
    float *smem;

    __device__ Gen(const GenArgs &a_, float *sm, int wave) : a(a_), smem(sm)
    {
        lane = threadIdx.x & 63;
        c = lane & 15;
        rg = lane >> 4;
        const int chain = wave / a.n_tiles;
        tile = wave % a.n_tiles;
        seq = chain / a.h_v;
        h = chain % a.h_v;
        hq = h / (a.h_v / a.h_qk);
        if (a.cu) {
            base = a.cu[seq];
            len = (long)a.cu[seq + 1] - base;
        } else {
            base = (long)seq * a.T;
            len = a.T;
        }
        nb = (int)((len + a.L - 1) / a.L);
    }
    __device__ __forceinline__ int col() const { return tile * 16 + c; }
    __device__ __forceinline__ long ck_group0() const
    {
        const long nblk = ((long)a.T + a.L - 1) / a.L;
        return a.cu ? a.ck_off[seq] : (long)seq * ((nblk + kStride - 1) / kStride);
    }
    // state tile addresses: global [d_k][d_v] layout (row i, this lane's column)
    __device__ __forceinline__ float *ckpt_ptr(long grp) const
    {
        return a.ckpt + ((grp * a.h_v + h) * (long)DK) * a.dv + col();
    }
    __device__ __forceinline__ void ld_state(float (&S)[NR], const float *p) const
    {
#pragma unroll
        for (int m = 0; m < NR; ++m) S[m] = p[(long)(rg * NR + m) * a.dv];
    }
    __device__ __forceinline__ void st_state(float *p, const float (&S)[NR]) const
    {
#pragma unroll
        for (int m = 0; m < NR; ++m) p[(long)(rg * NR + m) * a.dv] = S[m];
    }
    __device__ __forceinline__ void lds_put(int slot, const float (&S)[NR]) const
    {
#pragma unroll
        for (int m = 0; m < NR; ++m) smem[(slot * NR + m) * 64 + lane] = S[m];
    }
    __device__ __forceinline__ void lds_get(float (&S)[NR], int slot) const
    {
#pragma unroll
        for (int m = 0; m < NR; ++m) S[m] = smem[(slot * NR + m) * 64 + lane];
    }
    __device__ __forceinline__ float *uslot(int t) const { return smem + (kMaxSpans + kSpan) * ST + t * 64; }

    // inputs of position r (absolute row) of stream st
    struct Tok {
        float k[NR];
        float v, alpha, beta;
    };
    __device__ __forceinline__ void load_tok(Tok &t, const GenStream &s, long r) const
    {
        load_row<NR>(t.k, static_cast<const In *>(s.k) + (r * a.h_qk + hq) * DK + rg * NR);
        t.v = ld1(static_cast<const In *>(s.v) + (r * a.h_v + h) * a.dv + col());
        t.alpha = expf(s.g[r * a.h_v + h]);
        t.beta = s.beta[r * a.h_v + h];
    }
    // one forward step; returns u of this lane's column
    __device__ __forceinline__ float fwd(float (&S)[NR], const Tok &t) const
    {
        float ks = 0.f;
#pragma unroll
        for (int m = 0; m < NR; ++m) ks = fmaf(t.k[m], S[m], ks);
        const float u = t.v - t.alpha * col_sum(ks);
        const float bu = t.beta * u;
#pragma unroll
        for (int m = 0; m < NR; ++m) S[m] = fmaf(t.alpha, S[m], t.k[m] * bu);
        return u;
    }
    // add a row vector (rows rg NR + m) summed over the tile's columns into dst[row]
    __device__ __forceinline__ void add_rows(float *dst, float (&x)[NR]) const
    {
        int row0;
        row_sums<NR>(x, c, row0);
#pragma unroll
        for (int j = 0; j < NR / 16; ++j) atomicAdd(dst + rg * NR + row0 + j, x[j]);
    }
    // one backward step: dS (gradient of the state after the step) -> gradient before it;
    // Sp: the state before the step, u from its forward
    __device__ __forceinline__ void bwd(float (&dS)[NR], const float (&Sp)[NR], const Tok &t, float u,
                                        const GenStream &s, long r) const
    {
        float w = 0.f;
#pragma unroll
        for (int m = 0; m < NR; ++m) w = fmaf(t.k[m], dS[m], w);
        w = col_sum(w);
        if (rg == 0) s.dv[(r * a.h_v + h) * a.dv + col()] = t.beta * w;
        float e[NR];
        float gg = 0.f;
#pragma unroll
        for (int m = 0; m < NR; ++m) {
            const float sh = t.alpha * Sp[m];
            e[m] = t.beta * (dS[m] * u - sh * w);
            const float dsh = dS[m] - t.beta * t.k[m] * w;
            gg = fmaf(dsh, sh, gg);
            dS[m] = t.alpha * dsh;
        }
        // dbeta: sum over columns of w u (each column once: row group 0)
        const float db = wave_sum(rg == 0 ? w * u : 0.f);
        const float dg = wave_sum(gg);
        if (lane == 0) {
            atomicAdd(s.db + r * a.h_v + h, db);
            atomicAdd(s.dg + r * a.h_v + h, dg);
        }
        add_rows(s.dk + (r * a.h_qk + hq) * DK, e);
    }

    // The backward of one block (n positions from row r0) of stream s seeded with S0:
    // clean (dS = the gradient at the block's end, per-position outputs) or noisy (the
    // block-end readout).  Leaves in dS the gradient of the seed.
    template <bool CLEAN>
    __device__ void block(float (&dS)[NR], const float (&S0)[NR], const GenStream &s, long r0, int n) const
    {
        float S[NR];
#pragma unroll
        for (int m = 0; m < NR; ++m) S[m] = S0[m];
        Tok t;
        // forward: the states before every kSpan-th position
        for (int i = 0; i < n; ++i) {
            if (i % kSpan == 0) lds_put(i / kSpan, S);
            load_tok(t, s, r0 + i);
            fwd(S, t);
        }
        if (!CLEAN) {
            // block-end readout: dS~ = s sum_l q_l do_l^T, dq_l = s S~ do_l
#pragma unroll
            for (int m = 0; m < NR; ++m) dS[m] = 0.f;
            for (int i = 0; i < n; ++i) {
                const long r = r0 + i;
                float q[NR], p[NR];
                load_row<NR>(q, static_cast<const In *>(s.q) + (r * a.h_qk + hq) * DK + rg * NR);
                const float d = a.scale * ld1(static_cast<const Out *>(s.dout) + (r * a.h_v + h) * a.dv + col());
#pragma unroll
                for (int m = 0; m < NR; ++m) {
                    dS[m] = fmaf(q[m], d, dS[m]);
                    p[m] = S[m] * d;
                }
                add_rows(s.dq + (r * a.h_qk + hq) * DK, p);
            }
        }
        // backward, span by span from the last
        for (int sp = (n - 1) / kSpan; sp >= 0; --sp) {
            const int i0 = sp * kSpan, i1 = i0 + kSpan < n ? i0 + kSpan : n;
            lds_get(S, sp);
            for (int i = i0; i < i1; ++i) {
                lds_put(kMaxSpans + (i - i0), S);
                load_tok(t, s, r0 + i);
                uslot(i - i0)[lane] = fwd(S, t);
            }
            // S: the state after position i1 - 1
            for (int i = i1 - 1; i >= i0; --i) {
                const long r = r0 + i;
                load_tok(t, s, r);
                if (CLEAN) {
                    float q[NR], p[NR];
                    load_row<NR>(q, static_cast<const In *>(s.q) + (r * a.h_qk + hq) * DK + rg * NR);
                    const float d = a.scale * ld1(static_cast<const Out *>(s.dout) + (r * a.h_v + h) * a.dv + col());
#pragma unroll
                    for (int m = 0; m < NR; ++m) {
                        dS[m] = fmaf(q[m], d, dS[m]);
                        p[m] = S[m] * d;
                    }
                    add_rows(s.dq + (r * a.h_qk + hq) * DK, p);
                }
                float Sp[NR];
                lds_get(Sp, kMaxSpans + (i - i0));
                bwd(dS, Sp, t, uslot(i - i0)[lane], s, r);
#pragma unroll
                for (int m = 0; m < NR; ++m) S[m] = Sp[m];
            }
        }
    }
};

// The clean state before every kStride-th block of each chain.
template <typename In, typename Out, int DK>
__global__ void __launch_bounds__(64) bdgdn_bwd_gen_ckpt_kernel(GenArgs a)
{
    extern __shared__ __align__(16) float gsm[];
    typedef Gen<In, Out, DK> G;
    G w(a, gsm, blockIdx.x);
    if (w.seq >= a.n_seq) return;
    float S[G::NR];
    if (a.h0)
        w.ld_state(S, a.h0 + ((long)w.seq * a.h_v + w.h) * DK * a.dv + w.col());
    else
#pragma unroll
        for (int m = 0; m < G::NR; ++m) S[m] = 0.f;
    const long g0 = w.ck_group0();
    typename G::Tok t;
    for (int b = 0; b < w.nb; ++b) {
        if (b % kStride == 0) w.st_state(w.ckpt_ptr(g0 + b / kStride), S);
        const long r0 = w.base + (long)b * a.L;
        const int n = (int)(w.len - (long)b * a.L < a.L ? w.len - (long)b * a.L : a.L);
        for (int i = 0; i < n; ++i) {
            w.load_tok(t, a.st[0], r0 + i);
            w.fwd(S, t);
        }
    }
}

// The backward walk of each chain.
template <typename In, typename Out, int DK>
__global__ void __launch_bounds__(64) bdgdn_bwd_gen_walk_kernel(GenArgs a)
{
    extern __shared__ __align__(16) float gsm[];
    typedef Gen<In, Out, DK> G;
    constexpr int NR = G::NR;
    G w(a, gsm, blockIdx.x);
    if (w.seq >= a.n_seq) return;
    float dS[NR];
    if (a.dht)
        w.ld_state(dS, a.dht + ((long)w.seq * a.h_v + w.h) * DK * a.dv + w.col());
    else
#pragma unroll
        for (int m = 0; m < NR; ++m) dS[m] = 0.f;
    float *scr = a.scratch + (long)blockIdx.x * kStride * DK * 16;   // [kStride][DK rows][16 columns]
    auto scr_put = [&](int i, const float (&S)[NR]) {
#pragma unroll
        for (int m = 0; m < NR; ++m) scr[((long)i * DK + w.rg * NR + m) * 16 + w.c] = S[m];
    };
    auto scr_get = [&](float (&S)[NR], int i) {
#pragma unroll
        for (int m = 0; m < NR; ++m) S[m] = scr[((long)i * DK + w.rg * NR + m) * 16 + w.c];
    };
    const long g0 = w.ck_group0();
    typename G::Tok t;
    for (int grp = w.nb > 0 ? (w.nb - 1) / kStride : -1; grp >= 0; --grp) {
        const int b0 = grp * kStride, b1 = b0 + kStride < w.nb ? b0 + kStride : w.nb;
        // the block-start states of the group
        float S[NR];
        w.ld_state(S, w.ckpt_ptr(g0 + grp));
        for (int b = b0; b < b1; ++b) {
            scr_put(b - b0, S);
            if (b + 1 < b1) {
                const long r0 = w.base + (long)b * a.L;
                for (int i = 0; i < a.L; ++i) {
                    w.load_tok(t, a.st[0], r0 + i);
                    w.fwd(S, t);
                }
            }
        }
        for (int b = b1 - 1; b >= b0; --b) {
            const long r0 = w.base + (long)b * a.L;
            const int n = (int)(w.len - (long)b * a.L < a.L ? w.len - (long)b * a.L : a.L);
            float S0[NR];
            scr_get(S0, b - b0);
            // the noisy blocks of every view: the gradient of their seed
            float dSeed[NR];
#pragma unroll
            for (int m = 0; m < NR; ++m) dSeed[m] = 0.f;
            for (int v = 1; v <= a.n_views; ++v) {
                float d[NR];
                w.template block<false>(d, S0, a.st[v], r0, n);
#pragma unroll
                for (int m = 0; m < NR; ++m) dSeed[m] += d[m];
            }
            // the clean block: from the gradient at its end to the gradient at its start
            w.template block<true>(dS, S0, a.st[0], r0, n);
#pragma unroll
            for (int m = 0; m < NR; ++m) dS[m] += dSeed[m];
        }
    }
    if (a.dh0) w.st_state(a.dh0 + ((long)w.seq * a.h_v + w.h) * DK * a.dv + w.col(), dS);
}

__global__ void __launch_bounds__(256) bdgdn_bwd_gen_zero_kernel(float *p, long n)
{
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) p[i] = 0.f;
}

template <typename In, typename Out, int DK>
hipError_t launch_gen(const GenArgs &a, hipStream_t s)
{
    typedef Gen<In, Out, DK> G;
    const unsigned waves = (unsigned)(a.n_seq * a.h_v * a.n_tiles);
    auto kc = bdgdn_bwd_gen_ckpt_kernel<In, Out, DK>;
    auto kw = bdgdn_bwd_gen_walk_kernel<In, Out, DK>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kw), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       G::BYTES);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kc, dim3(waves), dim3(64), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(kw, dim3(waves), dim3(64), G::BYTES, s, a);
    return hipGetLastError();
}

}  // namespace

size_t bwd_generic_workspace(int n_seq, long total_blocks, int h_v, int dk, int dv)
{
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t groups = (size_t)total_blocks / kStride + n_seq;   // ceil(nb / kStride) summed over chains
    const size_t waves = (size_t)n_seq * h_v * (dv / 16);
    return up(groups * h_v * dk * dv * 4) + up(waves * kStride * dk * 16 * 4);
}

bool bwd_generic_supported(bool f32_in, int dk, int dv, int L, int n_views)
{
    return (dk == 64 || dk == 128) && (dv == 64 || dv == 128) && L >= 1 && L <= (f32_in ? 32 : 64) &&
           n_views >= 1 && n_views < kGenStreams;
}

hipError_t launch_bwd_generic(bool f32_in, bool f32_out, const GenBwdCall &c, hipStream_t s)
{
    GenArgs a = {};
    auto stream = [](const void *q, const void *k, const void *v, const float *g, const float *beta, const void *dout,
                     float *dq, float *dk, float *dv, float *dg, float *db) {
        return GenStream{q, k, v, g, beta, dout, dq, dk, dv, dg, db};
    };
    a.st[0] = stream(c.q, c.k, c.v, c.g, c.beta, c.dout, c.dq, c.dk, c.dv, c.dg, c.db);
    a.st[1] = stream(c.qn, c.kn, c.vn, c.gn, c.betan, c.doutn, c.dqn, c.dkn, c.dvn, c.dgn, c.dbn);
    for (int i = 0; i < c.n_more; ++i) {
        const BwdView &w = c.more[i];
        a.st[2 + i] = stream(w.q, w.k, w.v, w.g, w.beta, w.dout, w.dq, w.dk, w.dv, w.dg, w.db);
    }
    a.n_views = 1 + c.n_more;
    if (!bwd_generic_supported(f32_in, c.d_k, c.d_v, c.L, a.n_views)) return hipErrorInvalidValue;
    a.cu = c.cu;
    a.n_seq = c.n_seq;
    a.h0 = c.h0;
    a.dht = c.dht;
    a.dh0 = c.dh0;
    a.T = c.T; a.L = c.L; a.h_qk = c.h_qk; a.h_v = c.h_v; a.dk = c.d_k; a.dv = c.d_v;
    a.n_tiles = c.d_v / 16;
    a.scale = c.scale;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    a.ckpt = static_cast<float *>(c.workspace);
    const size_t groups = (size_t)c.total_blocks / kStride + c.n_seq;
    a.scratch = reinterpret_cast<float *>(static_cast<unsigned char *>(c.workspace) + up(groups * c.h_v * c.d_k * c.d_v * 4));
    if (c.cu) {
        if (c.n_seq > kMaxOrder || !c.cu_host) return hipErrorInvalidValue;
        long acc = 0;
        for (int i = 0; i < c.n_seq; ++i) {
            a.ck_off[i] = (int)acc;
            const long nb = ((long)c.cu_host[i + 1] - c.cu_host[i] + c.L - 1) / c.L;
            acc += (nb + kStride - 1) / kStride;
        }
        a.ck_off[c.n_seq] = (int)acc;
    }
    // the gradients summed with atomics start from zero
    for (int i = 0; i < a.n_views + 1; ++i) {
        const GenStream &st = a.st[i];
        const long qk = (long)c.rows * c.h_qk * c.d_k, gv = (long)c.rows * c.h_v;
        float *const ptr[4] = {st.dq, st.dk, st.dg, st.db};
        const long cnt[4] = {qk, qk, gv, gv};
        for (int j = 0; j < 4; ++j) {
            hipLaunchKernelGGL(bdgdn_bwd_gen_zero_kernel, dim3(512), dim3(256), 0, s, ptr[j], cnt[j]);
            if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
        }
    }
#define BDGDN_CASE(IN, OUT, DK) return launch_gen<IN, OUT, DK>(a, s);
    if (f32_in) {
        if (c.d_k == 64) BDGDN_CASE(float, float, 64) else BDGDN_CASE(float, float, 128)
    }
    if (f32_out) {
        if (c.d_k == 64) BDGDN_CASE(__bf16, float, 64) else BDGDN_CASE(__bf16, float, 128)
    }
    if (c.d_k == 64) BDGDN_CASE(__bf16, __bf16, 64) else BDGDN_CASE(__bf16, __bf16, 128)
#undef BDGDN_CASE
}

}  // namespace bdgdn
