// conv_kernels.hip -- the two-stream 1D causal ShortConv in front of the GDR (Appendix
// "ShortConv under two-stream training", eq. short-conv-clean and eq. short-conv-noisy, in
// the fused form that selects each lag's stream in place), forward and backward, for gfx950.
//
//   clean  pre_t  = bias + sum_i w_i xc_(t-i)
//   noisy  pre~_l = bias + sum_i w_i z_(l,i),  z_(l,i) = xn_(l-i) if l-i lies in l's diffusion
//          block (blocks counted from the document start), else xc_(l-i)
//   y = act(pre), act = identity or silu;  reads before the document start are zero
//   (Appendix "Document-packed training", the ShortConv lag mask).
//
// Both kernels stream [rows][D] tensors and are bound by HBM bandwidth.  A workgroup is 4
// waves over 64 channel vectors (a lane owns one VB-byte vector of channels); wave w takes
// the w-th of four consecutive row ranges, and the workgroups are numbered so that
// consecutive ranges run on the same XCD (its own L2) -- a range's W-1 halo rows are its
// neighbour's tail.  Rows whose W lags all lie in their own diffusion block (all but W-1
// rows of a block) take a path without any masking: the noisy output reads the noisy
// stream only.  The conditions are wave-uniform (every lane of a wave is on the same row),
// so the choice is a scalar branch.
//
// Forward: a wave's range is a short tile, fully unrolled: the loads of the whole tile and
// its halo are issued at once and kept in registers.
//
// Backward (gather form, no atomics): a wave streams a longer range in chunks with the next
// chunk's loads in flight.  The pre-activation gradients gc(s), gn(s) are recomputed for
// the range's rows and the W-1 rows after it; dx and dxn of a row collect the gradients of
// the outputs that read it; the filter and bias gradients of the four ranges of a workgroup
// are summed in LDS and written as one partial per workgroup, which a second kernel adds up
// in a fixed order (deterministic results).
#include <math.h>

#include <mutex>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace bdgdn {

namespace {

// Tile shapes: rows per wave tile (forward), rows per thread and rows per prefetched chunk
// (backward), bytes of channels per lane.
constexpr int kFwdTN = 8, kFwdVB = 8;
constexpr int kBwdTR = 256, kBwdU = 4, kBwdVB = 4;

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// A lane's channel vector as raw bits, and its buffer load and store.
template <int VB> struct Lane;
template <> struct Lane<4> {
    typedef unsigned T;
    static __device__ __forceinline__ T ld(__amdgpu_buffer_rsrc_t r, int v, int s)
    {
        return __builtin_amdgcn_raw_buffer_load_b32(r, v, s, 0);
    }
    static __device__ __forceinline__ void st(T x, __amdgpu_buffer_rsrc_t r, int v, int s)
    {
        __builtin_amdgcn_raw_buffer_store_b32(x, r, v, s, 0);
    }
};
template <> struct Lane<8> {
    typedef u32x2 T;
    static __device__ __forceinline__ T ld(__amdgpu_buffer_rsrc_t r, int v, int s)
    {
        return __builtin_amdgcn_raw_buffer_load_b64(r, v, s, 0);
    }
    static __device__ __forceinline__ void st(T x, __amdgpu_buffer_rsrc_t r, int v, int s)
    {
        __builtin_amdgcn_raw_buffer_store_b64(x, r, v, s, 0);
    }
};
template <> struct Lane<16> {
    typedef u32x4 T;
    static __device__ __forceinline__ T ld(__amdgpu_buffer_rsrc_t r, int v, int s)
    {
        return __builtin_amdgcn_raw_buffer_load_b128(r, v, s, 0);
    }
    static __device__ __forceinline__ void st(T x, __amdgpu_buffer_rsrc_t r, int v, int s)
    {
        __builtin_amdgcn_raw_buffer_store_b128(x, r, v, s, 0);
    }
};

// silu(p) = p sigmoid(p) and its derivative s (1 + p (1 - s)), with the hardware
// reciprocal (1 ulp); p -> -inf gives 0 (the reciprocal of +inf), p -> +inf gives p.
__device__ __forceinline__ float sigm(float p) { return __builtin_amdgcn_rcpf(1.f + __expf(-p)); }
__device__ __forceinline__ float act_fwd(float p, int act) { return act ? p * sigm(p) : p; }
__device__ __forceinline__ float act_grad(float p, int act)
{
    if (!act) return 1.f;
    const float s = sigm(p);
    return s * fmaf(p, 1.f - s, 1.f);
}

template <typename In, int N, typename T> __device__ __forceinline__ void unpack(T raw, float (&v)[N])
{
    static_assert(sizeof(T) == N * sizeof(In), "lane vector size");
    In e[N];
    __builtin_memcpy(e, &raw, sizeof(T));
#pragma unroll
    for (int j = 0; j < N; ++j) v[j] = to_f(e[j]);
}
template <typename In, int N, typename T> __device__ __forceinline__ T pack(const float (&v)[N])
{
    In e[N];
#pragma unroll
    for (int j = 0; j < N; ++j) e[j] = to_e<In>(v[j]);
    T raw;
    __builtin_memcpy(&raw, e, sizeof(T));
    return raw;
}

// Row access through a buffer resource whose base is the first row a wave touches: the
// per-lane channel offset is the one vector register of the address and the row offset is
// a scalar, so a tile's loads cost no address registers.  Callers clamp every row into
// [base, rows) themselves.
template <int VB> struct Rows {
    __amdgpu_buffer_rsrc_t r;
    __device__ Rows(const void *p, long row0, long rows, int row_bytes)
    {
        const long n = (rows - row0) * row_bytes;
        r = __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(static_cast<const char *>(p)) + row0 * row_bytes,
                                              (short)0, (int)(n < 0x7fffffffL ? n : 0x7fffffffL), 0x00020000);
    }
    __device__ __forceinline__ typename Lane<VB>::T ld(int voff, int soff) const { return Lane<VB>::ld(r, voff, soff); }
    __device__ __forceinline__ void st(typename Lane<VB>::T x, int voff, int soff) const
    {
        Lane<VB>::st(x, r, voff, soff);
    }
};

// Logical workgroup id: the hardware hands workgroup b to XCD b % 8, so ids b = 8k + x of
// the first 8 * (G / 8) workgroups become x * (G / 8) + k (a contiguous range per XCD);
// the remainder keeps its id.
__device__ __forceinline__ int xcd_id(int b, int G)
{
    const int full = G & ~7;
    if (b >= full) return b;
    return (b & 7) * (full >> 3) + (b >> 3);
}

// The document [ds, de) and diffusion block [bs, be) of a row, started at a tile's first row
// and then stepped one row at a time, so that a step only tests for the row reaching the
// end of its block or document.  Packed: documents from cu (possibly empty ones); otherwise
// sequences of seqlen rows.  Rows fit in 32 bits (the host checks B * T).  All fields are
// wave-uniform.
struct Cursor {
    int ds, de, bs, be, d;
    __device__ void start(const ConvArgs &a, int t)
    {
        if (a.cu) {
            int lo = 0, hi = a.n_docs;   // the last d < n_docs with cu[d] <= t
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (a.cu[mid] <= t)
                    lo = mid;
                else
                    hi = mid;
            }
            d = lo;
            ds = a.cu[lo];
            de = a.cu[lo + 1];
        } else {
            d = t / a.seqlen;
            ds = d * a.seqlen;
            de = ds + a.seqlen;
        }
        bs = ds + (t - ds) / a.L * a.L;
        be = bs + a.L;
    }
    // t = the previous row + 1
    __device__ __forceinline__ void step(const ConvArgs &a, int t)
    {
        if (t == be) {   // next block of the document (it may run past the document's end)
            bs = be;
            be += a.L;
        }
        if (t == de) {   // next non-empty document
            do {
                ++d;
                ds = a.cu ? a.cu[d] : d * a.seqlen;
                de = a.cu ? a.cu[d + 1] : ds + a.seqlen;
            } while (t >= de);
            bs = ds;
            be = ds + a.L;
        }
    }
};

// Pre-activations of row t from its lag window: xc[i], xn[i] hold rows t - i of x, xn.
template <int W, int N>
__device__ __forceinline__ void pre_of(int t, const Cursor &c, const float (&xc)[W][N], const float (&xn)[W][N],
                                       const float (&w)[N][W], const float (&b)[N], float (&pc)[N], float (&pn)[N])
{
#pragma unroll
    for (int j = 0; j < N; ++j) pc[j] = pn[j] = b[j];
    if (t - (W - 1) >= c.bs) {   // every lag in t's block: clean reads clean, noisy reads noisy
#pragma unroll
        for (int i = 0; i < W; ++i)
#pragma unroll
            for (int j = 0; j < N; ++j) {
                pc[j] = fmaf(w[j][i], xc[i][j], pc[j]);
                pn[j] = fmaf(w[j][i], xn[i][j], pn[j]);
            }
        return;
    }
#pragma unroll
    for (int i = 0; i < W; ++i) {
        const int src = t - i;
        if (src < c.ds) break;   // this lag and the later ones fall before the document
        const bool in_blk = src >= c.bs;
#pragma unroll
        for (int j = 0; j < N; ++j) {
            pc[j] = fmaf(w[j][i], xc[i][j], pc[j]);
            pn[j] = fmaf(w[j][i], in_blk ? xn[i][j] : xc[i][j], pn[j]);
        }
    }
}

template <int W, int N>
__device__ __forceinline__ void load_filter(const ConvArgs &a, int c0, float (&w)[N][W], float (&b)[N])
{
#pragma unroll
    for (int j = 0; j < N; ++j) {
#pragma unroll
        for (int i = 0; i < W; ++i) w[j][i] = a.w[(c0 + j) * W + i];
        b[j] = a.bias ? a.bias[c0 + j] : 0.f;
    }
}

}  // namespace

template <typename In, int W, int TN, int VB>
__global__ void __launch_bounds__(256) bdgdn_shortconv_fwd_kernel(ConvArgs a)
{
    constexpr int N = VB / (int)sizeof(In);
    constexpr int R = TN + W - 1;   // rows t0 - W + 1 .. t0 + TN - 1
    typedef typename Lane<VB>::T T;
    const int lane = threadIdx.x & 63, wave = wave_id();
    const int lid = xcd_id(blockIdx.x, gridDim.x);
    const int cv = lid / a.n_rg * 64 + lane;
    const int rows = (int)a.rows;
    const int t0 = ((lid % a.n_rg) * 4 + wave) * TN;
    if (cv * N >= a.D || t0 >= rows) return;
    const int c0 = cv * N;
    const int rb = a.D * (int)sizeof(In), voff = c0 * (int)sizeof(In);
    // input rows t0 - W + 1 .. t0 + TN - 1, clamped into [b0, rows) (clamped rows are never used)
    const int b0 = t0 - (W - 1) > 0 ? t0 - (W - 1) : 0;
    const Rows<VB> gx(a.x, b0, rows, rb), gxn(a.xn, b0, rows, rb);
    T rx[R], rn[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        int src = t0 - (W - 1) + r;
        src = src < b0 ? b0 : (src >= rows ? rows - 1 : src);
        const int so = (int)(src - b0) * rb;
        rx[r] = gx.ld(voff, so);
        rn[r] = gxn.ld(voff, so);
    }
    float w[N][W], b[N];
    load_filter<W, N>(a, c0, w, b);
    const Rows<VB> gy(a.y, t0, rows, rb), gyn(a.yn, t0, rows, rb);
    Cursor cur;
    cur.start(a, t0);
#pragma unroll
    for (int u = 0; u < TN; ++u) {
        const int t = t0 + u;
        if (t >= rows) break;
        if (u > 0) cur.step(a, t);
        float lx[W][N], ln[W][N];   // rows t - i
#pragma unroll
        for (int i = 0; i < W; ++i) {
            unpack<In>(rx[u + W - 1 - i], lx[i]);
            unpack<In>(rn[u + W - 1 - i], ln[i]);
        }
        float pc[N], pn[N];
        pre_of<W, N>(t, cur, lx, ln, w, b, pc, pn);
#pragma unroll
        for (int j = 0; j < N; ++j) {
            pc[j] = act_fwd(pc[j], a.act);
            pn[j] = act_fwd(pn[j], a.act);
        }
        gy.st(pack<In, N, T>(pc), voff, u * rb);
        gyn.st(pack<In, N, T>(pn), voff, u * rb);
    }
}

// Backward over a thread's TR rows [t0, t1), streamed in chunks of UW rows (the smallest
// multiple of W that is at least U): the loads of the next chunk (x, xn, dy, dyn) are issued
// before the current chunk is computed.  The last W rows of x, xn (the lag window) and the
// pending dx, dxn of the last W rows stay in registers in circular slots: row s lives in
// slot (s - t0) mod W, which is a constant inside the unrolled chunk (UW is a multiple of W),
// so rows never move between registers.  Reader rows run to t1 + W - 2 (the W - 1 rows after
// the range read its last rows); rows before t0 are the previous range's, so what this thread
// gathers for them is dropped.
template <typename In, int W, int TR, int U, int VB>
__global__ void __launch_bounds__(256) bdgdn_shortconv_bwd_kernel(ConvArgs a)
{
    constexpr int N = VB / (int)sizeof(In);
    constexpr int P = N * (W + 1);   // filter + bias gradients per thread
    constexpr int UW = (U + W - 1) / W * W;
    typedef typename Lane<VB>::T T;
    __shared__ float red[3][P][64];
    const int lane = threadIdx.x & 63, wave = wave_id();
    const int lid = xcd_id(blockIdx.x, gridDim.x);
    const int cg = lid / a.n_rg, rg = lid % a.n_rg;
    const int cv = cg * 64 + lane;
    const int rows = (int)a.rows;
    const int t0 = (rg * 4 + wave) * TR;
    const bool live = cv * N < a.D && t0 < rows;   // idle threads still join the reduction
    float gw[N][W], gb[N];
#pragma unroll
    for (int j = 0; j < N; ++j) {
        gb[j] = 0.f;
#pragma unroll
        for (int i = 0; i < W; ++i) gw[j][i] = 0.f;
    }
    if (live) {
        const int c0 = cv * N;
        const int t1 = t0 + TR < rows ? t0 + TR : rows;
        const int s_end = t1 + W - 1 < rows ? t1 + W - 1 : rows;   // one past the last reader
        const int rb = a.D * (int)sizeof(In), voff = c0 * (int)sizeof(In);
        const int b0 = t0 - (W - 1) > 0 ? t0 - (W - 1) : 0;
        const Rows<VB> gx(a.x, b0, rows, rb), gxn(a.xn, b0, rows, rb);
        const Rows<VB> gdy(a.dy, t0, rows, rb), gdyn(a.dyn, t0, rows, rb);
        const Rows<VB> gdx(a.y, t0, rows, rb), gdxn(a.yn, t0, rows, rb);
        float w[N][W], b[N];
        load_filter<W, N>(a, c0, w, b);
        // lag window: slot (s - t0) mod W holds row s of x, xn (clamped rows before 0 are
        // masked as lying before the document)
        float wx[W][N], wn[W][N];
#pragma unroll
        for (int k = 1; k < W; ++k) {
            const int src = t0 - k < b0 ? b0 : t0 - k;
            unpack<In>(gx.ld(voff, (src - b0) * rb), wx[W - k]);
            unpack<In>(gxn.ld(voff, (src - b0) * rb), wn[W - k]);
        }
        // pending input gradients of the last W rows, in the same slots
        float ac[W][N], an[W][N];
#pragma unroll
        for (int k = 0; k < W; ++k)
#pragma unroll
            for (int j = 0; j < N; ++j) ac[k][j] = an[k][j] = 0.f;
        T cx[UW], cn[UW], cy[UW], cyn[UW];
        auto load_chunk = [&](int s0, T (&lx)[UW], T (&ln)[UW], T (&ly)[UW], T (&lyn)[UW]) {
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                // rows from the last reader on are never used: they re-read the last one (a
                // cache hit) rather than fetch a row of the next range
                const int s = s0 + u < s_end ? s0 + u : s_end - 1;
                lx[u] = gx.ld(voff, (s - b0) * rb);
                ln[u] = gxn.ld(voff, (s - b0) * rb);
                ly[u] = gdy.ld(voff, (s - t0) * rb);
                lyn[u] = gdyn.ld(voff, (s - t0) * rb);
            }
        };
        load_chunk(t0, cx, cn, cy, cyn);
        Cursor cur;
        cur.start(a, t0);
        // one chunk of UW rows from s0; TAIL: rows past the range (reader rows of its last
        // rows, which count for no filter gradient) and the end of the readers
        auto chunk = [&](int s0, auto tail) {
            constexpr bool TAIL = decltype(tail)::value;
            T nx[UW], nn[UW], ny[UW], nyn[UW];
            // the next chunk, unless this is the last one (a tail chunk can be)
            const bool next = !TAIL || s0 + UW < s_end;
            if (next) load_chunk(s0 + UW, nx, nn, ny, nyn);
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                const int s = s0 + u;
                if (TAIL && s >= s_end) break;
                const int sl = u % W;                       // slot of row s
                unpack<In>(cx[u], wx[sl]);
                unpack<In>(cn[u], wn[sl]);
                if (s > t0) cur.step(a, s);
                // lag i of row s sits in slot (u - i) mod W
                float lx[W][N], ln[W][N];
#pragma unroll
                for (int i = 0; i < W; ++i)
#pragma unroll
                    for (int j = 0; j < N; ++j) {
                        lx[i][j] = wx[(u - i + W * UW) % W][j];
                        ln[i][j] = wn[(u - i + W * UW) % W][j];
                    }
                float pc[N], pn[N], gc[N], gn[N];
                pre_of<W, N>(s, cur, lx, ln, w, b, pc, pn);
                unpack<In>(cy[u], gc);
                unpack<In>(cyn[u], gn);
#pragma unroll
                for (int j = 0; j < N; ++j) {
                    gc[j] *= act_grad(pc[j], a.act);
                    gn[j] *= act_grad(pn[j], a.act);
                }
                const bool own = !TAIL || s < t1;   // this range's output: counts for the filter and bias
                if (s - (W - 1) >= cur.bs) {   // every lag in s's block
#pragma unroll
                    for (int i = 0; i < W; ++i) {
                        const int li = (u - i + W * UW) % W;
#pragma unroll
                        for (int j = 0; j < N; ++j) {
                            ac[li][j] = fmaf(w[j][i], gc[j], ac[li][j]);
                            an[li][j] = fmaf(w[j][i], gn[j], an[li][j]);
                        }
                        if (own)
#pragma unroll
                            for (int j = 0; j < N; ++j)
                                gw[j][i] = fmaf(gn[j], ln[i][j], fmaf(gc[j], lx[i][j], gw[j][i]));
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < W; ++i) {
                        if (s - i < cur.ds) break;   // before the document: nothing read
                        const int li = (u - i + W * UW) % W;
                        const bool in_blk = s - i >= cur.bs;
                        if (in_blk) {
#pragma unroll
                            for (int j = 0; j < N; ++j) {
                                ac[li][j] = fmaf(w[j][i], gc[j], ac[li][j]);
                                an[li][j] = fmaf(w[j][i], gn[j], an[li][j]);
                            }
                        } else {
#pragma unroll
                            for (int j = 0; j < N; ++j) ac[li][j] = fmaf(w[j][i], gc[j] + gn[j], ac[li][j]);
                        }
                        if (own)
#pragma unroll
                            for (int j = 0; j < N; ++j)
                                gw[j][i] = fmaf(gn[j], in_blk ? ln[i][j] : lx[i][j], fmaf(gc[j], lx[i][j], gw[j][i]));
                    }
                }
                if (own)
#pragma unroll
                    for (int j = 0; j < N; ++j) gb[j] += gc[j] + gn[j];
                // row s - (W - 1) (slot (u + 1) mod W) has seen its last reader; its slot
                // becomes row s + 1's
                const int done = s - (W - 1);
                const int ds = (u + 1) % W;
                if (done >= t0) {
                    gdx.st(pack<In, N, T>(ac[ds]), voff, (done - t0) * rb);
                    gdxn.st(pack<In, N, T>(an[ds]), voff, (done - t0) * rb);
                }
#pragma unroll
                for (int j = 0; j < N; ++j) ac[ds][j] = an[ds][j] = 0.f;
            }
            if (next)
#pragma unroll
                for (int u = 0; u < UW; ++u) {
                    cx[u] = nx[u];
                    cn[u] = nn[u];
                    cy[u] = ny[u];
                    cyn[u] = nyn[u];
                }
        };
        int s0 = t0;
        for (; s0 + UW <= t1; s0 += UW) chunk(s0, std::false_type());
        for (; s0 < s_end; s0 += UW) chunk(s0, std::true_type());
        // rows of the range whose readers ran past the end of the tensor: rows s_end - k,
        // k = 1 .. W - 1, in slots (s_end - k - t0) mod W
#pragma unroll
        for (int k = 1; k < W; ++k) {
            const int d = s_end - k;
            if (d >= t0 && d < t1) {
                const int sl = (d - t0) % W;
#pragma unroll
                for (int q = 0; q < W; ++q)
                    if (q == sl) {
                        gdx.st(pack<In, N, T>(ac[q]), voff, (d - t0) * rb);
                        gdxn.st(pack<In, N, T>(an[q]), voff, (d - t0) * rb);
                    }
            }
        }
    }
    // waves 1..3 hand their sums to wave 0, which writes the workgroup's partial,
    // laid out [group][W + 1][D] (slot W is the bias)
    if (wave > 0)
#pragma unroll
        for (int j = 0; j < N; ++j) {
#pragma unroll
            for (int i = 0; i < W; ++i) red[wave - 1][j * (W + 1) + i][lane] = gw[j][i];
            red[wave - 1][j * (W + 1) + W][lane] = gb[j];
        }
    __syncthreads();
    if (wave == 0 && cv * N < a.D) {
        float *p = a.part + (long)rg * (W + 1) * a.D + cv * N;
#pragma unroll
        for (int i = 0; i <= W; ++i) {
            float o[N];
#pragma unroll
            for (int j = 0; j < N; ++j) {
                const int k = j * (W + 1) + i;
                o[j] = (i < W ? gw[j][i] : gb[j]) + red[0][k][lane] + red[1][k][lane] + red[2][k][lane];
            }
#pragma unroll
            for (int j = 0; j < N; ++j) p[(long)i * a.D + j] = o[j];
        }
    }
}

// dw, dbias: the workgroups' partials summed in a fixed order (eight interleaved running
// sums, so that eight loads are in flight, then added pairwise); one thread per (slot,
// channel).
template <int W>
__global__ void __launch_bounds__(256) bdgdn_shortconv_reduce_kernel(ConvArgs a)
{
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= (W + 1) * a.D) return;
    const long stride = (long)(W + 1) * a.D;
    const float *p = a.part + e;
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int g = 0;
    for (; g + 8 <= a.n_rg; g += 8)
#pragma unroll
        for (int u = 0; u < 8; ++u) s[u] += p[(g + u) * stride];
    for (int u = 0; g < a.n_rg; ++g, ++u) s[u] += p[g * stride];
    const float acc = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
    const int i = e / a.D, c = e % a.D;
    if (i < W)
        a.dw[c * W + i] = acc;
    else if (a.dbias)
        a.dbias[c] = acc;
}

static int row_groups(long rows, int tn) { return (int)((rows + 4 * tn - 1) / (4 * tn)); }

size_t conv_part_floats(long rows, int D, int width) { return (size_t)row_groups(rows, kBwdTR) * (width + 1) * D; }

namespace {

template <typename In, int VB> unsigned conv_grid(const ConvArgs &a)
{
    const long ncg = (a.D / (VB / (int)sizeof(In)) + 63) / 64;
    return (unsigned)(ncg * a.n_rg);
}

template <typename In, int W> hipError_t fwd_w(ConvArgs a, hipStream_t s)
{
    a.n_rg = row_groups(a.rows, kFwdTN);
    if (a.rows == 0) return hipSuccess;
    hipLaunchKernelGGL((bdgdn_shortconv_fwd_kernel<In, W, kFwdTN, kFwdVB>), dim3(conv_grid<In, kFwdVB>(a)), dim3(256),
                       0, s, a);
    return hipGetLastError();
}

template <typename In, int W> hipError_t bwd_w(ConvArgs a, hipStream_t s)
{
    a.n_rg = row_groups(a.rows, kBwdTR);
    if (a.rows > 0) {
        hipLaunchKernelGGL((bdgdn_shortconv_bwd_kernel<In, W, kBwdTR, kBwdU, kBwdVB>), dim3(conv_grid<In, kBwdVB>(a)),
                           dim3(256), 0, s, a);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((bdgdn_shortconv_reduce_kernel<W>), dim3(((W + 1) * a.D + 255) / 256), dim3(256), 0, s, a);
    return hipGetLastError();
}

#define BDGDN_CONV_WIDTHS(FN, IN)            \
    switch (width) {                         \
    case 1: return FN<IN, 1>(a, s);          \
    case 2: return FN<IN, 2>(a, s);          \
    case 3: return FN<IN, 3>(a, s);          \
    case 4: return FN<IN, 4>(a, s);          \
    default: return hipErrorInvalidValue;    \
    }

}  // namespace

hipError_t launch_shortconv_fwd(bool bf16, int width, const ConvArgs &a, hipStream_t s)
{
    if (bf16) {
        BDGDN_CONV_WIDTHS(fwd_w, __bf16)
    }
    BDGDN_CONV_WIDTHS(fwd_w, float)
}

hipError_t launch_shortconv_bwd(bool bf16, int width, const ConvArgs &a, hipStream_t s)
{
    if (bf16) {
        BDGDN_CONV_WIDTHS(bwd_w, __bf16)
    }
    BDGDN_CONV_WIDTHS(bwd_w, float)
}

#undef BDGDN_CONV_WIDTHS

// The fixed scratch of the no-allocation backward: the per-workgroup dw / dbias partials,
// in device memory the library holds for the life of the process (each GPU it runs on has
// its own copy at its own address).  Every partial slot a launch reads is written by that
// launch first, so nothing needs clearing between calls.  On the host this name is only a
// stand-in for the device symbol: host code uses the address conv_noalloc_scratch returns.
static __device__ __align__(256) float scratch[kConvScratchBytes / sizeof(float)];

hipError_t conv_noalloc_scratch(hipStream_t stream, float **ptr)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static float *addr[kMaxDevices] = {};
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    int dev = cur;
    if (stream) {
        e = hipStreamGetDevice(stream, &dev);
        if (e != hipSuccess) return e;
    }
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        // the symbol's address on `dev`, looked up once with that device current
        if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (dev != cur) {
            const hipError_t r = hipSetDevice(cur);
            if (e == hipSuccess) e = r;
        }
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = static_cast<float *>(p);
    }
    *ptr = addr[dev];
    return hipSuccess;
}

}  // namespace bdgdn
