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
 *   - the backward of the two-stream training forward (Appendix "Backward primitives":
 *     the per-step backward, eq. per-step-bwd, applied token by token in reverse; the
 *     noisy block's block-end readout, eq. noisy-readout-bwd, followed by its reverse sweep
 *     with zero per-step output gradient; and the block-level chain rule,
 *     eq. dh-block-recursion: the gradient at a noisy block's seed is added to the clean
 *     state gradient at the end of the previous block).
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
 * Forward of one block from state S_in over rows [p0, p1) (clean or noisy inputs),
 * keeping what the per-step backward needs: Sst[i] = the state after step i (Sst[-1] is
 * S_in, passed separately), Spre[i] = exp(g) times the state before step i, uu[i] = the
 * prediction error v - S_pre^T k (before the step size).
 */
static void block_states(const dims_t *d, long p0, long p1, int h, const double *S_in,
                         const double *k, const double *v, const double *g, const double *beta,
                         double *Spre, double *Sst, double *uu)
{
    const size_t ssz = (size_t)d->dk * d->dv;
    for (long t = p0; t < p1; ++t) {
        const long i = t - p0;
        const double *prev = i == 0 ? S_in : Sst + (i - 1) * ssz;
        const double alpha = exp(gate_at(g, d, t, h)), b = gate_at(beta, d, t, h);
        const double *kt = row_qk(k, d, t, h), *vt = row_v(v, d, t, h);
        double *sp = Spre + i * ssz, *st = Sst + i * ssz, *ut = uu + i * d->dv;
        for (size_t e = 0; e < ssz; ++e) sp[e] = alpha * prev[e];
        for (int j = 0; j < d->dv; ++j) {
            double acc = 0.0;
            for (int a = 0; a < d->dk; ++a) acc += sp[a * d->dv + j] * kt[a];
            ut[j] = vt[j] - acc;
        }
        for (int a = 0; a < d->dk; ++a)
            for (int j = 0; j < d->dv; ++j) st[a * d->dv + j] = sp[a * d->dv + j] + kt[a] * b * ut[j];
    }
}

/*
 * Eq. per-step-bwd for one token: dS holds dL/dS_t on entry and dL/dS_(t-1) on exit.
 * do_ may be NULL (a noisy step: its output gradient entered through the block-end
 * readout).  Gradients are added into dq, dk (d_k vectors), dv (d_v) and *dg, *db.
 */
static void per_step_bwd(const dims_t *d, double *dS, const double *do_, const double *q, const double *k,
                         double g, double beta, const double *Spre, const double *St, const double *u,
                         double *dq, double *dk, double *dv, double *dg, double *db, double *ddelta)
{
    const int dkk = d->dk, dvv = d->dv;
    if (do_) {
        for (int a = 0; a < dkk; ++a) {              /* dq = s S_t do */
            double acc = 0.0;
            for (int j = 0; j < dvv; ++j) acc += St[a * dvv + j] * do_[j];
            dq[a] += d->scale * acc;
        }
        for (int a = 0; a < dkk; ++a)                /* dS_t += s q do^T */
            for (int j = 0; j < dvv; ++j) dS[a * dvv + j] += d->scale * q[a] * do_[j];
    }
    for (int j = 0; j < dvv; ++j) {                  /* d delta = dS_t^T k */
        double acc = 0.0;
        for (int a = 0; a < dkk; ++a) acc += dS[a * dvv + j] * k[a];
        ddelta[j] = acc;
    }
    for (int a = 0; a < dkk; ++a) {                  /* dk_write = dS_t delta, delta = beta u */
        double acc = 0.0;
        for (int j = 0; j < dvv; ++j) acc += dS[a * dvv + j] * beta * u[j];
        dk[a] += acc;
    }
    double dbeta = 0.0;
    for (int j = 0; j < dvv; ++j) {                  /* du = beta d delta; dv = du; dbeta = d delta . u */
        dbeta += ddelta[j] * u[j];
        ddelta[j] *= beta;                           /* ddelta now holds du */
        dv[j] += ddelta[j];
    }
    *db += dbeta;
    for (int a = 0; a < dkk; ++a) {                  /* dk_pred = -S_pre du */
        double acc = 0.0;
        for (int j = 0; j < dvv; ++j) acc += Spre[a * dvv + j] * ddelta[j];
        dk[a] -= acc;
    }
    double dgate = 0.0;
    const double decay = exp(g);
    for (int a = 0; a < dkk; ++a)                    /* dS_pre = dS_t - k du^T; dg = <dS_pre, S_pre> */
        for (int j = 0; j < dvv; ++j) {
            const double dsp = dS[a * dvv + j] - k[a] * ddelta[j];
            dgate += dsp * Spre[a * dvv + j];
            dS[a * dvv + j] = decay * dsp;           /* dS_(t-1) = exp(g) dS_pre */
        }
    *dg += dgate;
}

typedef struct {
    double *dq, *dk, *dv, *dg, *db;
} grads_t;

static double *grow_qk(double *base, const dims_t *d, long row, int h)
{
    return base + ((size_t)row * d->h_qk + h / (d->h_v / d->h_qk)) * d->dk;
}

/*
 * Backward of two_stream_unit over rows [r0, r1), one v-head.  dS holds dL/d(final clean
 * state) on entry (dht or zero) and dL/d(initial state) on exit (dh0).  ck: clean states
 * before every block (filled here by a forward pass from S_init).
 */
static void two_stream_unit_bwd(const dims_t *d, int L, long r0, long r1, int h, const double *S_init,
                                const double *q, const double *k, const double *v, const double *g,
                                const double *beta, const double *qn, const double *kn, const double *vn,
                                const double *gn, const double *betan, const double *do_, const double *don,
                                grads_t gc, grads_t gnz, double *dS, double *ck, double *Spre, double *Sst,
                                double *uu, double *dSn, double *tmp)
{
    const size_t ssz = (size_t)d->dk * d->dv;
    const long nblk = (r1 - r0 + L - 1) / L;
    /* checkpoints: the clean state before each block */
    memcpy(ck, S_init, ssz * sizeof(double));
    for (long b = 0; b + 1 < nblk; ++b) {
        const long p0 = r0 + b * L, p1 = p0 + L;
        block_states(d, p0, p1, h, ck + b * ssz, k, v, g, beta, Spre, Sst, uu);
        memcpy(ck + (b + 1) * ssz, Sst + (p1 - p0 - 1) * ssz, ssz * sizeof(double));
    }
    for (long b = nblk - 1; b >= 0; --b) {
        const long p0 = r0 + b * L, p1 = p0 + L < r1 ? p0 + L : r1;
        const double *seed = ck + b * ssz;
        /* clean block, tokens in reverse */
        block_states(d, p0, p1, h, seed, k, v, g, beta, Spre, Sst, uu);
        for (long t = p1 - 1; t >= p0; --t) {
            const long i = t - p0;
            per_step_bwd(d, dS, row_v(do_, d, t, h), row_qk(q, d, t, h), row_qk(k, d, t, h), gate_at(g, d, t, h),
                         gate_at(beta, d, t, h), Spre + i * ssz, Sst + i * ssz, uu + i * d->dv,
                         grow_qk(gc.dq, d, t, h), grow_qk(gc.dk, d, t, h), gc.dv + ((size_t)t * d->h_v + h) * d->dv,
                         gc.dg + (size_t)t * d->h_v + h, gc.db + (size_t)t * d->h_v + h, tmp);
        }
        /* noisy block b from the same seed: block-end readout, then the reverse sweep */
        block_states(d, p0, p1, h, seed, kn, vn, gn, betan, Spre, Sst, uu);
        const double *Send = Sst + (p1 - p0 - 1) * ssz;
        memset(dSn, 0, ssz * sizeof(double));
        for (long l = p0; l < p1; ++l) {
            const double *ql = row_qk(qn, d, l, h), *dol = row_v(don, d, l, h);
            double *dql = grow_qk(gnz.dq, d, l, h);
            for (int a = 0; a < d->dk; ++a) {
                double acc = 0.0;
                for (int j = 0; j < d->dv; ++j) {
                    acc += Send[a * d->dv + j] * dol[j];             /* dq~ = s S~_end do~ */
                    dSn[a * d->dv + j] += d->scale * ql[a] * dol[j]; /* dS~_end = s sum q~ do~^T */
                }
                dql[a] += d->scale * acc;
            }
        }
        for (long l = p1 - 1; l >= p0; --l) {
            const long i = l - p0;
            per_step_bwd(d, dSn, NULL, NULL, row_qk(kn, d, l, h), gate_at(gn, d, l, h), gate_at(betan, d, l, h),
                         Spre + i * ssz, Sst + i * ssz, uu + i * d->dv, NULL, grow_qk(gnz.dk, d, l, h),
                         gnz.dv + ((size_t)l * d->h_v + h) * d->dv, gnz.dg + (size_t)l * d->h_v + h,
                         gnz.db + (size_t)l * d->h_v + h, tmp);
        }
        /* eq. dh-block-recursion: the seed is the clean state at the end of block b - 1 */
        for (size_t e = 0; e < ssz; ++e) dS[e] += dSn[e];
    }
}

/*
 * oracle_bwd_train: gradients of  sum <do, o> + sum <don, on> + <dht, ht>  with respect to
 * every input of oracle_fwd_train (same layouts; dq, dk, dqn, dkn per q/k head summed over
 * its v-heads).  dht and dh0 may be NULL (zero / not wanted); h0 NULL means zero.
 * Work is split over (sequence, q/k head) units so that grouped v-heads accumulate into
 * their q/k head's gradients in one thread.
 */
int oracle_bwd_train(int B, int T, int n_seqs, const int32_t *cu,
                     int h_qk, int h_v, int dk, int dv, int L, double scale,
                     const double *q, const double *k, const double *v, const double *g, const double *beta,
                     const double *qn, const double *kn, const double *vn, const double *gn, const double *betan,
                     const double *h0, const double *do_, const double *don, const double *dht,
                     double *dq, double *dkk, double *dvv, double *dg, double *db,
                     double *dqn, double *dkn, double *dvn, double *dgn, double *dbn, double *dh0)
{
    if (L < 1 || h_qk < 1 || h_v < 1 || h_v % h_qk || dk < 1 || dv < 1) return -1;
    dims_t d = {h_qk, h_v, dk, dv, scale};
    const int nseq = cu ? n_seqs : B;
    const long rows = cu ? cu[n_seqs] : (long)B * T;
    const size_t ssz = (size_t)dk * dv;
    long maxlen = 0;
    for (int n = 0; n < nseq; ++n) {
        const long len = cu ? cu[n + 1] - cu[n] : T;
        if (len > maxlen) maxlen = len;
    }
    const long maxblk = (maxlen + L - 1) / L + 1;
    memset(dq, 0, (size_t)rows * h_qk * dk * sizeof(double));
    memset(dkk, 0, (size_t)rows * h_qk * dk * sizeof(double));
    memset(dvv, 0, (size_t)rows * h_v * dv * sizeof(double));
    memset(dg, 0, (size_t)rows * h_v * sizeof(double));
    memset(db, 0, (size_t)rows * h_v * sizeof(double));
    memset(dqn, 0, (size_t)rows * h_qk * dk * sizeof(double));
    memset(dkn, 0, (size_t)rows * h_qk * dk * sizeof(double));
    memset(dvn, 0, (size_t)rows * h_v * dv * sizeof(double));
    memset(dgn, 0, (size_t)rows * h_v * sizeof(double));
    memset(dbn, 0, (size_t)rows * h_v * sizeof(double));
    const grads_t gc = {dq, dkk, dvv, dg, db}, gz = {dqn, dkn, dvn, dgn, dbn};
    const long nunits = (long)nseq * h_qk;
    const int group = h_v / h_qk;
    int err = 0;
#pragma omp parallel
    {
        double *S0 = malloc(ssz * sizeof(double)), *dS = malloc(ssz * sizeof(double));
        double *ck = malloc(maxblk * ssz * sizeof(double));
        double *Spre = malloc((size_t)L * ssz * sizeof(double)), *Sst = malloc((size_t)L * ssz * sizeof(double));
        double *uu = malloc((size_t)L * dv * sizeof(double)), *dSn = malloc(ssz * sizeof(double));
        double *tmp = malloc((size_t)dv * sizeof(double));
        const int ok = S0 && dS && ck && Spre && Sst && uu && dSn && tmp;
        if (!ok) {
#pragma omp atomic write
            err = -2;
        }
#pragma omp for schedule(dynamic, 1)
        for (long unit = 0; unit < nunits; ++unit) {
            if (!ok) continue;
            const int n = (int)(unit / h_qk), hq = (int)(unit % h_qk);
            const long r0 = cu ? cu[n] : (long)n * T, r1 = cu ? cu[n + 1] : (long)n * T + T;
            for (int h = hq * group; h < (hq + 1) * group; ++h) {
                const size_t so = ((size_t)n * h_v + h) * ssz;
                if (h0) memcpy(S0, h0 + so, ssz * sizeof(double));
                else memset(S0, 0, ssz * sizeof(double));
                if (dht) memcpy(dS, dht + so, ssz * sizeof(double));
                else memset(dS, 0, ssz * sizeof(double));
                if (r1 > r0)
                    two_stream_unit_bwd(&d, L, r0, r1, h, S0, q, k, v, g, beta, qn, kn, vn, gn, betan, do_, don,
                                        gc, gz, dS, ck, Spre, Sst, uu, dSn, tmp);
                if (dh0) memcpy(dh0 + so, dS, ssz * sizeof(double));
            }
        }
        free(S0); free(dS); free(ck); free(Spre); free(Sst); free(uu); free(dSn); free(tmp);
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
