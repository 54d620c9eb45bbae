/*
 * bdgdn_oracle.c -- plain, slow, sequential fp64 reference of the block-diffusion
 * Gated Delta Rule (FLARE, arXiv 2606.01774).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code, header,
 * table or helper with the HIP library; nothing in the product links it.
 *
 * What it computes, and where the paper defines it:
 *   - one GDR step in the expanded per-step form (Appendix, "Per-step recurrence",
 *     eq. per-step-fwd): S_pre = exp(g) S; u = v - S_pre^T k; delta = beta u;
 *     S = S_pre + k delta^T; o = s S^T q.
 *   - the two-stream schedule (Sec. 3.2, eq. flare-gdn-schedule): the clean stream is the
 *     causal recurrence; noisy block b is seeded with the clean state after the last
 *     clean token before the block, runs its own L updates, and every position of
 *     the block reads the block-end noisy state (block-end readout, Appendix
 *     eq. noisy-block-fwd).
 *   - document packing (Appendix "Document-packed training"): each document is
 *     an independent sequence; the state starts from zero (or the caller's h0) at
 *     each document start; the last block of a document may be partial.
 *   - serving passes (Appendix "Diffusion-Trust Sampling", "Differences between the
 *     denoise pass and the state-update pass"): denoise reads the cached state and
 *     never writes it; commit runs the token-causal pass and writes the state back;
 *     the AR-Trust verify pass also keeps the states at the verify positions, and the
 *     accept step writes the state at each request's accepted offset back to the pool
 *     (Appendix "Serving-system machinery", cache-and-scatter).
 *   - the two-stream 1D causal ShortConv feeding the GDR, forward and backward
 *     (Appendix "ShortConv under two-stream training").
 *
 * Layouts (row = token index in the flattened [B*T] or packed token axis):
 *   q,k  [row][h_qk][d_k]    v,o [row][h_v][d_v]    g,beta [row][h_v]
 *   states [unit][h_v][d_k][d_v] (paper orientation: S is d_k x d_v, o = s S^T q)
 *   v-head h reads q/k head h / (h_v / h_qk).
 * All arrays are fp64.  Parallelism: OpenMP over independent (sequence, v-head) units.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One step of eq. per-step-fwd on S (dk x dv, row-major). u is dv scratch. */
static void gdr_step(double *S, int dk, int dv, const double *k, const double *v,
                     double g, double beta, double *u)
{
    const double alpha = exp(g);                       /* gating decay */
    for (int i = 0; i < dk * dv; ++i) S[i] *= alpha;    /* S_pre = alpha S */
    for (int j = 0; j < dv; ++j) {                      /* u = v - S_pre^T k */
        double acc = 0.0;
        for (int i = 0; i < dk; ++i) acc += S[i * dv + j] * k[i];
        u[j] = beta * (v[j] - acc);                     /* delta = beta u */
    }
    for (int i = 0; i < dk; ++i)                        /* S = S_pre + k delta^T */
        for (int j = 0; j < dv; ++j) S[i * dv + j] += k[i] * u[j];
}

/* o = s S^T q */
static void readout(const double *S, int dk, int dv, const double *q, double scale, double *o)
{
    for (int j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (int i = 0; i < dk; ++i) acc += S[i * dv + j] * q[i];
        o[j] = scale * acc;
    }
}

typedef struct {
    int h_qk, h_v, dk, dv;
    double scale;
} dims_t;

static const double *row_qk(const double *base, const dims_t *d, long row, int h)
{
    int hq = h / (d->h_v / d->h_qk);
    return base + ((size_t)row * d->h_qk + hq) * d->dk;
}
static const double *row_v(const double *base, const dims_t *d, long row, int h)
{
    return base + ((size_t)row * d->h_v + h) * d->dv;
}
static double *row_o(double *base, const dims_t *d, long row, int h)
{
    return base + ((size_t)row * d->h_v + h) * d->dv;
}
static double gate_at(const double *base, const dims_t *d, long row, int h)
{
    return base[(size_t)row * d->h_v + h];
}

/*
 * Two-stream training forward over rows [r0, r1) of one document, one v-head.
 * S (dk x dv) holds the clean state on entry (h0 or zero) and on exit (ht).
 */
static void two_stream_unit(const dims_t *d, int L, long r0, long r1, int h,
                            const double *q, const double *k, const double *v,
                            const double *g, const double *beta,
                            const double *qn, const double *kn, const double *vn,
                            const double *gn, const double *betan,
                            double *o, double *on, double *S, double *Sn, double *u)
{
    const size_t ssz = (size_t)d->dk * d->dv;
    for (long p0 = r0; p0 < r1; p0 += L) {
        long p1 = p0 + L < r1 ? p0 + L : r1;
        /* noisy block: seed with the clean state after the last token before p0 */
        memcpy(Sn, S, ssz * sizeof(double));
        for (long l = p0; l < p1; ++l)
            gdr_step(Sn, d->dk, d->dv, row_qk(kn, d, l, h), row_v(vn, d, l, h),
                     gate_at(gn, d, l, h), gate_at(betan, d, l, h), u);
        for (long l = p0; l < p1; ++l)       /* block-end readout */
            readout(Sn, d->dk, d->dv, row_qk(qn, d, l, h), d->scale, row_o(on, d, l, h));
        /* clean stream: causal steps with per-token readout */
        for (long t = p0; t < p1; ++t) {
            gdr_step(S, d->dk, d->dv, row_qk(k, d, t, h), row_v(v, d, t, h),
                     gate_at(g, d, t, h), gate_at(beta, d, t, h), u);
            readout(S, d->dk, d->dv, row_qk(q, d, t, h), d->scale, row_o(o, d, t, h));
        }
    }
}

/*
 * oracle_fwd_train: both streams.  Non-packed: cu == NULL, batch B sequences of T rows.
 * Packed: cu = [n_seqs+1] offsets into a single packed token axis (B must be 1).
 * h0 / ht: [n_units_seq][h_v][dk][dv] or NULL.
 */
int oracle_fwd_train(int B, int T, int n_seqs, const int32_t *cu,
                     int h_qk, int h_v, int dk, int dv, int L, double scale,
                     const double *q, const double *k, const double *v,
                     const double *g, const double *beta,
                     const double *qn, const double *kn, const double *vn,
                     const double *gn, const double *betan,
                     const double *h0, double *o, double *on, double *ht)
{
    if (L < 1 || h_qk < 1 || h_v < 1 || h_v % h_qk || dk < 1 || dv < 1) return -1;
    dims_t d = {h_qk, h_v, dk, dv, scale};
    const int nseq = cu ? n_seqs : B;
    const long nunits = (long)nseq * h_v;
    const size_t ssz = (size_t)dk * dv;
    int err = 0;
#pragma omp parallel
    {
        double *S = malloc(ssz * sizeof(double));
        double *Sn = malloc(ssz * sizeof(double));
        double *u = malloc((size_t)dv * sizeof(double));
        const int ok = S && Sn && u;
        if (!ok) {
#pragma omp atomic write
            err = -2;
        }
        /* every thread reaches the worksharing loop; one without buffers skips its units */
#pragma omp for schedule(dynamic, 1)
        for (long unit = 0; unit < nunits; ++unit) {
            if (ok) {
                int n = (int)(unit / h_v), h = (int)(unit % h_v);
                long r0 = cu ? cu[n] : (long)n * T;
                long r1 = cu ? cu[n + 1] : (long)n * T + T;
                if (h0) memcpy(S, h0 + ((size_t)n * h_v + h) * ssz, ssz * sizeof(double));
                else memset(S, 0, ssz * sizeof(double));
                two_stream_unit(&d, L, r0, r1, h, q, k, v, g, beta, qn, kn, vn, gn, betan,
                                o, on, S, Sn, u);
                if (ht) memcpy(ht + ((size_t)n * h_v + h) * ssz, S, ssz * sizeof(double));
            }
        }
        free(S); free(Sn); free(u);
    }
    return err;
}

/*
 * oracle_denoise: R requests, each a block of L noisy tokens ([R][L] rows).
 * The seed of request r is pool[slot[r]] (slot == NULL means slot[r] = r); the
 * pool is read, never written.  o receives the block-end readout of every position.
 */
int oracle_denoise(int R, int h_qk, int h_v, int dk, int dv, int L, double scale,
                   const double *pool, const int32_t *slot,
                   const double *q, const double *k, const double *v,
                   const double *g, const double *beta, double *o)
{
    if (L < 1 || h_qk < 1 || h_v < 1 || h_v % h_qk) return -1;
    dims_t d = {h_qk, h_v, dk, dv, scale};
    const size_t ssz = (size_t)dk * dv;
    const long nunits = (long)R * h_v;
    int err = 0;
#pragma omp parallel
    {
        double *Sn = malloc(ssz * sizeof(double));
        double *u = malloc((size_t)dv * sizeof(double));
        const int ok = Sn && u;
        if (!ok) {
#pragma omp atomic write
            err = -2;
        }
#pragma omp for schedule(dynamic, 1)
        for (long unit = 0; unit < nunits; ++unit) {
            if (!ok) continue;
            int r = (int)(unit / h_v), h = (int)(unit % h_v);
            int s = slot ? slot[r] : r;
            memcpy(Sn, pool + ((size_t)s * h_v + h) * ssz, ssz * sizeof(double));
            for (long l = (long)r * L; l < (long)r * L + L; ++l)
                gdr_step(Sn, dk, dv, row_qk(k, &d, l, h), row_v(v, &d, l, h),
                         gate_at(g, &d, l, h), gate_at(beta, &d, l, h), u);
            for (long l = (long)r * L; l < (long)r * L + L; ++l)
                readout(Sn, dk, dv, row_qk(q, &d, l, h), scale, row_o(o, &d, l, h));
        }
        free(Sn); free(u);
    }
    return err;
}

/*
 * oracle_commit: the token-causal state-update pass.  pool[slot[r]] is advanced by
 * the L tokens of request r and written back; o (optional) gets the causal readout.
 */
int oracle_commit(int R, int h_qk, int h_v, int dk, int dv, int L, double scale,
                  double *pool, const int32_t *slot,
                  const double *q, const double *k, const double *v,
                  const double *g, const double *beta, double *o)
{
    if (L < 1 || h_qk < 1 || h_v < 1 || h_v % h_qk) return -1;
    dims_t d = {h_qk, h_v, dk, dv, scale};
    const size_t ssz = (size_t)dk * dv;
    const long nunits = (long)R * h_v;
    int err = 0;
#pragma omp parallel
    {
        double *u = malloc((size_t)dv * sizeof(double));
        const int ok = u != NULL;
        if (!ok) {
#pragma omp atomic write
            err = -2;
        }
#pragma omp for schedule(dynamic, 1)
        for (long unit = 0; unit < nunits; ++unit) {
            if (!ok) continue;
            int r = (int)(unit / h_v), h = (int)(unit % h_v);
            int s = slot ? slot[r] : r;
            double *S = pool + ((size_t)s * h_v + h) * ssz;
            for (long t = (long)r * L; t < (long)r * L + L; ++t) {
                gdr_step(S, dk, dv, row_qk(k, &d, t, h), row_v(v, &d, t, h),
                         gate_at(g, &d, t, h), gate_at(beta, &d, t, h), u);
                if (o) readout(S, dk, dv, row_qk(q, &d, t, h), scale, row_o(o, &d, t, h));
            }
        }
        free(u);
    }
    return err;
}

/*
 * oracle_commit_record: the commit pass that also keeps the verify-position states
 * (Appendix "Serving-system machinery for the hybrid backbone", cache-and-scatter, and
 * Algorithm "AR-Trust serving round"): before the update of block position
 * p = L - n_rec + i (i = 0 .. n_rec-1) the current state is copied to
 * states[r][i][h] (layout [R][n_rec][h_v][dk][dv]); the pool then holds the state after
 * all L positions, as after oracle_commit.
 */
int oracle_commit_record(int R, int h_qk, int h_v, int dk, int dv, int L, int n_rec, double scale,
                         double *pool, const int32_t *slot,
                         const double *q, const double *k, const double *v,
                         const double *g, const double *beta, double *o, double *states)
{
    if (L < 1 || h_qk < 1 || h_v < 1 || h_v % h_qk || n_rec < 1 || n_rec > L) return -1;
    dims_t d = {h_qk, h_v, dk, dv, scale};
    const size_t ssz = (size_t)dk * dv;
    const long nunits = (long)R * h_v;
    int err = 0;
#pragma omp parallel
    {
        double *u = malloc((size_t)dv * sizeof(double));
        const int ok = u != NULL;
        if (!ok) {
#pragma omp atomic write
            err = -2;
        }
#pragma omp for schedule(dynamic, 1)
        for (long unit = 0; unit < nunits; ++unit) {
            if (!ok) continue;
            int r = (int)(unit / h_v), h = (int)(unit % h_v);
            int s = slot ? slot[r] : r;
            double *S = pool + ((size_t)s * h_v + h) * ssz;
            for (int p = 0; p < L; ++p) {
                const long t = (long)r * L + p;
                const int i = p - (L - n_rec);
                if (i >= 0)   /* the state before position p */
                    memcpy(states + (((size_t)r * n_rec + i) * h_v + h) * ssz, S, ssz * sizeof(double));
                gdr_step(S, dk, dv, row_qk(k, &d, t, h), row_v(v, &d, t, h),
                         gate_at(g, &d, t, h), gate_at(beta, &d, t, h), u);
                if (o) readout(S, dk, dv, row_qk(q, &d, t, h), scale, row_o(o, &d, t, h));
            }
        }
        free(u);
    }
    return err;
}

/*
 * oracle_accept_states: the gather-scatter after a verify decision.  Request r keeps
 * the state at its accepted offset: pool[slot[r]][h] = states[r][accept[r]][h] for
 * accept[r] < n_rec; accept[r] == n_rec keeps the state already in the pool.
 */
int oracle_accept_states(int R, int h_v, int dk, int dv, int n_rec, double *pool, const int32_t *slot,
                         const double *states, const int32_t *accept)
{
    if (h_v < 1 || n_rec < 1) return -1;
    for (int r = 0; r < R; ++r)
        if (accept[r] < 0 || accept[r] > n_rec) return -1;
    const size_t ssz = (size_t)dk * dv;
    for (int r = 0; r < R; ++r) {
        if (accept[r] == n_rec) continue;
        const int s = slot ? slot[r] : r;
        for (int h = 0; h < h_v; ++h)
            memcpy(pool + ((size_t)s * h_v + h) * ssz,
                   states + (((size_t)r * n_rec + accept[r]) * h_v + h) * ssz, ssz * sizeof(double));
    }
    return 0;
}

/*
 * The two-stream 1D causal ShortConv (Appendix "ShortConv under two-stream training",
 * eq. short-conv-clean and eq. short-conv-noisy) for one packed axis of rows:
 *   clean  pre_t  = bias + sum_i w_i * xc_(t-i)
 *   noisy  pre~_l = bias + sum_i w_i * z_(l,i),  z_(l,i) = xn_(l-i) if l-i >= the start of
 *          l's diffusion block, else xc_(l-i)
 *   y = act(pre): act 0 = identity, 1 = silu (x / (1 + exp(-x)))
 * depthwise over D channels (w [D][W], w[c][i] = the lag-i weight), every read outside the
 * current document (before its start) contributing zero; documents and blocks as in the
 * training schedule (blocks counted from each document start).  x, xn, y, yn: [rows][D].
 */
static double act_of(double p, int act) { return act ? p / (1.0 + exp(-p)) : p; }
static double act_grad(double p, int act)
{
    if (!act) return 1.0;
    const double sg = 1.0 / (1.0 + exp(-p));
    return sg * (1.0 + p * (1.0 - sg));
}

/* pre-activations of one position of both streams (doc starts at row a) */
static void conv_pre(long t, long a, int L, int D, int W, int c, const double *x, const double *xn,
                     const double *w, const double *bias, double *pc, double *pn)
{
    const long blk = a + ((t - a) / L) * L;   /* start of t's diffusion block */
    double sc = bias ? bias[c] : 0.0, sn = sc;
    for (int i = 0; i < W; ++i) {
        const long src = t - i;
        if (src < a) break;
        sc += w[c * W + i] * x[src * D + c];
        sn += w[c * W + i] * (src >= blk ? xn[src * D + c] : x[src * D + c]);
    }
    *pc = sc;
    *pn = sn;
}

int oracle_shortconv_fwd(int n_docs, const int32_t *cu, int D, int W, int L, int act,
                         const double *x, const double *xn, const double *w, const double *bias,
                         double *y, double *yn)
{
    if (n_docs < 1 || D < 1 || W < 1 || L < 1) return -1;
    for (int d = 0; d < n_docs; ++d)
        for (long t = cu[d]; t < cu[d + 1]; ++t)
            for (int c = 0; c < D; ++c) {
                double pc, pn;
                conv_pre(t, cu[d], L, D, W, c, x, xn, w, bias, &pc, &pn);
                y[t * D + c] = act_of(pc, act);
                yn[t * D + c] = act_of(pn, act);
            }
    return 0;
}

/*
 * Backward of oracle_shortconv_fwd: given dy, dyn, the gradients of the loss with respect
 * to x, xn, w and bias (dx, dxn, dw [D][W], dbias [D], all overwritten), by the chain rule
 * through every read of the forward: each output's pre-activation gradient
 * dpre = dy act'(pre) is sent to the input it read at each lag (the clean or the noisy
 * stream, as chosen in the forward) times that lag's weight, and to w and bias.
 */
int oracle_shortconv_bwd(int n_docs, const int32_t *cu, int D, int W, int L, int act,
                         const double *x, const double *xn, const double *w, const double *bias,
                         const double *dy, const double *dyn, double *dx, double *dxn, double *dw,
                         double *dbias)
{
    if (n_docs < 1 || D < 1 || W < 1 || L < 1) return -1;
    const long rows = cu[n_docs];
    memset(dx, 0, (size_t)rows * D * sizeof(double));
    memset(dxn, 0, (size_t)rows * D * sizeof(double));
    memset(dw, 0, (size_t)D * W * sizeof(double));
    if (dbias) memset(dbias, 0, (size_t)D * sizeof(double));
    for (int d = 0; d < n_docs; ++d) {
        const long a = cu[d];
        for (long t = a; t < cu[d + 1]; ++t)
            for (int c = 0; c < D; ++c) {
                double pc, pn;
                conv_pre(t, a, L, D, W, c, x, xn, w, bias, &pc, &pn);
                const double gc = dy[t * D + c] * act_grad(pc, act);
                const double gn = dyn[t * D + c] * act_grad(pn, act);
                if (dbias) dbias[c] += gc + gn;
                const long blk = a + ((t - a) / L) * L;
                for (int i = 0; i < W; ++i) {
                    const long src = t - i;
                    if (src < a) break;
                    dx[src * D + c] += w[c * W + i] * gc;
                    dw[c * W + i] += gc * x[src * D + c];
                    if (src >= blk) {
                        dxn[src * D + c] += w[c * W + i] * gn;
                        dw[c * W + i] += gn * xn[src * D + c];
                    } else {
                        dx[src * D + c] += w[c * W + i] * gn;
                        dw[c * W + i] += gn * x[src * D + c];
                    }
                }
            }
    }
    return 0;
}

void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
