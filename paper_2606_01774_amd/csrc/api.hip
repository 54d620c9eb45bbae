// api.hip -- the C ABI (include/bdgdn.h): host-side validation, scheduling and
// dispatch.  Nothing here allocates device memory or synchronises the host.
#include <math.h>

#include <algorithm>
#include <numeric>
#include <vector>

#include "bdgdn.h"
#include "bwd.hpp"
#include "kernels.hpp"

using namespace bdgdn;

namespace {

int lp_of(int L) { return L <= 16 ? 16 : (L <= 32 ? 32 : 64); }

bool dims_ok(int d) { return d == 64 || d == 128; }

// Token tensors are read and written with 16-byte vector accesses.
bool aligned16(const void *p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// (dtype, out_dtype) -> element types of the kernels; false if not offered.
bool types_of(int dtype, int out_dtype, Types &ty)
{
    if (dtype == BDGDN_BF16 && out_dtype == BDGDN_F32) { ty = Types::BF16_IN_F32_OUT; return true; }
    if (dtype == BDGDN_BF16 && out_dtype == BDGDN_BF16) { ty = Types::BF16_IN_BF16_OUT; return true; }
    if (dtype == BDGDN_F32 && out_dtype == BDGDN_F32) { ty = Types::F32; return true; }
    return false;
}

// Shared validation of head shapes and dtypes.  Returns a status.
int check_heads(int h_qk, int h_v, int d_k, int d_v, int block, float scale, int dtype, int out_dtype)
{
    if (h_qk <= 0 || h_v <= 0 || d_k <= 0 || d_v <= 0 || block <= 0) return BDGDN_ERR_INVALID_ARG;
    if (h_v % h_qk != 0) return BDGDN_ERR_INVALID_ARG;
    if (!isfinite(scale)) return BDGDN_ERR_INVALID_ARG;
    Types ty;
    if (!types_of(dtype, out_dtype, ty)) return BDGDN_ERR_UNSUPPORTED;
    if (!dims_ok(d_k) || !dims_ok(d_v) || block > 64) return BDGDN_ERR_UNSUPPORTED;
    if (!fwd_supported(ty, d_k, lp_of(block))) return BDGDN_ERR_UNSUPPORTED;
    return BDGDN_OK;
}

// Validation of a training descriptor and its packing (Appendix "Document-packed
// training": document starts are block-aligned; the tail may be partial).
int check_fwd(const bdgdn_fwd_desc_t *d, const int32_t *cu_dev, const int32_t *cu_host)
{
    if (!d) return BDGDN_ERR_INVALID_ARG;
    int st = check_heads(d->h_qk, d->h_v, d->d_k, d->d_v, d->block, d->scale, d->dtype, d->out_dtype);
    if (st != BDGDN_OK) return st;
    if (d->batch <= 0 || d->seqlen < 0 || d->num_seqs < 0) return BDGDN_ERR_INVALID_ARG;
    if (d->route != BDGDN_ROUTE_FUSED && d->route != BDGDN_ROUTE_SPLIT && d->route != BDGDN_ROUTE_ONEPASS &&
        d->route != BDGDN_ROUTE_RECORDS && d->route != BDGDN_ROUTE_CHUNKED)
        return BDGDN_ERR_INVALID_ARG;
    if ((long)d->batch * d->seqlen > 0x7fffffffL) return BDGDN_ERR_UNSUPPORTED;
    const bool packed = d->num_seqs > 0;
    if (packed != (cu_dev != nullptr) || packed != (cu_host != nullptr)) return BDGDN_ERR_INVALID_ARG;
    if (packed) {
        if (d->batch != 1) return BDGDN_ERR_INVALID_ARG;
        if (cu_host[0] != 0 || cu_host[d->num_seqs] != d->seqlen) return BDGDN_ERR_INVALID_ARG;
        for (int i = 0; i < d->num_seqs; ++i)
            if (cu_host[i + 1] < cu_host[i]) return BDGDN_ERR_INVALID_ARG;
        for (int i = 0; i < d->num_seqs; ++i)
            if (cu_host[i] % d->block != 0) return BDGDN_ERR_UNALIGNED;
    }
    if (d->route == BDGDN_ROUTE_SPLIT) {
        Types ty;
        types_of(d->dtype, d->out_dtype, ty);
        if (!split_supported(ty, d->d_k, d->d_v, lp_of(d->block))) return BDGDN_ERR_UNSUPPORTED;
    }
    if (d->route == BDGDN_ROUTE_CHUNKED) {
        Types ty;
        types_of(d->dtype, d->out_dtype, ty);
        if (!chunked_supported(ty, d->d_k, d->d_v, lp_of(d->block)) || d->num_seqs > kMaxOrder)
            return BDGDN_ERR_UNSUPPORTED;
    }
    return BDGDN_OK;
}

// Validation of a ShortConv descriptor and its packing.  Blocks are counted from each
// document start, so document starts need no alignment.
int check_conv(const bdgdn_conv_desc_t *d, const int32_t *cu_dev, const int32_t *cu_host)
{
    if (!d) return BDGDN_ERR_INVALID_ARG;
    if (d->batch <= 0 || d->seqlen < 0 || d->num_seqs < 0 || d->channels <= 0 || d->block <= 0)
        return BDGDN_ERR_INVALID_ARG;
    if (d->activation != BDGDN_ACT_NONE && d->activation != BDGDN_ACT_SILU) return BDGDN_ERR_INVALID_ARG;
    if (d->dtype != BDGDN_BF16 && d->dtype != BDGDN_F32) return BDGDN_ERR_UNSUPPORTED;
    if (d->width < 1 || d->width > 4) return BDGDN_ERR_UNSUPPORTED;
    if (d->channels % (d->dtype == BDGDN_BF16 ? 4 : 2) != 0) return BDGDN_ERR_UNSUPPORTED;
    if ((long)d->batch * d->seqlen > 0x7fffffffL) return BDGDN_ERR_UNSUPPORTED;
    const bool packed = d->num_seqs > 0;
    if (packed != (cu_dev != nullptr) || packed != (cu_host != nullptr)) return BDGDN_ERR_INVALID_ARG;
    if (packed) {
        if (d->batch != 1) return BDGDN_ERR_INVALID_ARG;
        if (cu_host[0] != 0 || cu_host[d->num_seqs] != d->seqlen) return BDGDN_ERR_INVALID_ARG;
        for (int i = 0; i < d->num_seqs; ++i)
            if (cu_host[i + 1] < cu_host[i]) return BDGDN_ERR_INVALID_ARG;
    }
    return BDGDN_OK;
}

bool aligned8(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 7) == 0; }

ConvArgs conv_args(const bdgdn_conv_desc_t *d, const int32_t *cu_dev, const void *x, const void *xn,
                   const float *w, const float *bias, void *y, void *yn)
{
    ConvArgs a = {};
    a.x = x; a.xn = xn; a.w = w; a.bias = bias; a.y = y; a.yn = yn;
    a.cu = d->num_seqs > 0 ? cu_dev : nullptr;
    a.rows = (long)d->batch * d->seqlen;
    a.D = d->channels; a.L = d->block; a.act = d->activation;
    a.n_docs = d->num_seqs; a.seqlen = d->seqlen;
    return a;
}

}  // namespace

extern "C" {

int32_t bdgdn_version(void) { return (0 << 16) | 1; }

const char *bdgdn_status_string(int status)
{
    switch (status) {
    case BDGDN_OK: return "ok";
    case BDGDN_ERR_INVALID_ARG: return "invalid argument";
    case BDGDN_ERR_UNSUPPORTED: return "unsupported size, dtype or route";
    case BDGDN_ERR_UNALIGNED: return "document start not aligned to the diffusion block";
    case BDGDN_ERR_WORKSPACE: return "workspace too small";
    case BDGDN_ERR_LAUNCH: return "kernel launch failed";
    case BDGDN_ERR_SCRATCH: return "input larger than the fixed scratch of the no-allocation entry point";
    default: return "unknown status";
    }
}

// Blocks of the packed axis (packed) or of all sequences: the UT records are indexed by
// (block, v-head); document starts are block-aligned, so blocks never straddle documents.
static long total_blocks(const bdgdn_fwd_desc_t *d)
{
    const long nblk = (d->seqlen + d->block - 1) / d->block;
    return d->num_seqs > 0 ? nblk : nblk * d->batch;
}

// Blocks of 34 .. 64 positions (even) run the one-kernel forward on two sub-blocks of half
// the block each.
static bool pair_blocks(const bdgdn_fwd_desc_t *d, Types ty)
{
    return !pipelined_supported(ty, d->d_k, lp_of(d->block)) && pair_supported(ty, d->d_k, d->block);
}

// Blocks of 1, 2, 4 or 8 positions run the one-kernel forward on 32-position clean chunks
// that hold several noisy blocks each (the noisy seeds inside a chunk are formed on chip).
static bool small_blocks(const bdgdn_fwd_desc_t *d, Types ty) { return small_supported(ty, d->d_k, d->block); }

// The fused route runs as one kernel where it can, else through the UT records.
static bool one_kernel(const bdgdn_fwd_desc_t *d, Types ty)
{
    return d->route == BDGDN_ROUTE_FUSED &&
           (pipelined_supported(ty, d->d_k, lp_of(d->block)) || pair_blocks(d, ty));
}

// The one-kernel forward on a descriptor's chains: the sub-block is the block, or half of
// it for pairs, or a 32-position chunk of small blocks (with the clean outputs only: a
// further noisy view keeps one block per step).
static hipError_t launch_one_kernel(const bdgdn_fwd_desc_t *d, Types ty, ScanArgs sa, hipStream_t s,
                                    bool clean_out = true)
{
    if (clean_out && small_blocks(d, ty)) {
        sa.nl = d->block;
        sa.L = 32;
        sa.nblk = (d->seqlen + 31) / 32;
        return launch_fwd_pipelined_small(ty, d->d_k, sa, s);
    }
    if (!pair_blocks(d, ty)) return launch_fwd_pipelined(ty, d->d_k, lp_of(d->block), sa, s, clean_out);
    sa.L = d->block / 2;
    sa.nblk = (d->seqlen + sa.L - 1) / sa.L;
    return launch_fwd_pipelined_pair(ty, d->d_k, sa, s, clean_out);
}

// The chunk-parallel schedule's plan: each chain (sequence or document, v-head) is cut
// into d_v tiles (one, or 32-column tiles when there are fewer chains than compute units)
// and into segments of G blocks, G the largest power of two (at least 16) that still
// gives every compute unit of the GPU a (chain, tile, segment) of its own; with enough
// chains and tiles a chain is one segment and there is no state pass.
constexpr int kComputeUnits = 256;
struct ChunkPlan {
    int tiles, G;
};
static ChunkPlan chunk_plan(const bdgdn_fwd_desc_t *d)
{
    const long chains = (long)(d->num_seqs > 0 ? d->num_seqs : d->batch) * d->h_v;
    ChunkPlan p;
    p.tiles = chains >= kComputeUnits ? 1 : d->d_v / 32;
    const long work = total_blocks(d) * d->h_v * p.tiles;   // (block, v-head, tile) triples
    const long nblk = (d->seqlen + d->block - 1) / d->block;
    // G: the largest power of two from 16 on with at least two (chain, segment, tile)
    // workgroups per compute unit and fewer blocks than a chain
    long G = 16;
    while (2 * G * 2 * kComputeUnits <= work && 2 * G < nblk) G *= 2;
    p.G = (int)G;
    return p;
}
static int chunk_segment(const bdgdn_fwd_desc_t *d) { return chunk_plan(d).G; }

// The fused route with at least as many chains as compute units: one workgroup per chain
// covering all d_v columns (the chunk-parallel schedule's output pass with one segment per
// chain, so no state pass and no workspace) instead of one per (chain, 32-column tile),
// which would repeat the d_v-independent work of every block once per tile.
static bool fused_uses_wide_pass(const bdgdn_fwd_desc_t *d, Types ty)
{
    const long chains = (long)(d->num_seqs > 0 ? d->num_seqs : d->batch) * d->h_v;
    return chunked_supported(ty, d->d_k, d->d_v, lp_of(d->block)) && d->num_seqs <= kMaxOrder &&
           chains >= kComputeUnits && !small_blocks(d, ty);
}
// Workspace of the chunk-parallel schedule: a clean UT record per (block, v-head) and a
// state per (segment start after the first, v-head), both bounded by the descriptor alone
// (a chain of nb blocks has ceil(nb / G) - 1 <= nb / G later segment starts).
struct ChunkLayout {
    size_t rec, ckpt, total;
};
static ChunkLayout chunk_layout(const bdgdn_fwd_desc_t *d)
{
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t blocks = (size_t)total_blocks(d);
    ChunkLayout l;
    l.rec = 0;
    l.ckpt = up(blocks * d->h_v * chunk_rec_bytes(lp_of(d->block)));
    l.total = l.ckpt + up((blocks / chunk_segment(d)) * d->h_v * (size_t)d->d_k * d->d_v * 4);
    return l;
}

static size_t workspace_bytes_of(const bdgdn_fwd_desc_t *d)
{
    Types ty;
    types_of(d->dtype, d->out_dtype, ty);
    if (d->route == BDGDN_ROUTE_CHUNKED) {
        if (!chunked_supported(ty, d->d_k, d->d_v, lp_of(d->block))) return 0;
        // every chain (at most nblk blocks) one segment: no state pass, no workspace
        if (chunk_segment(d) >= (d->seqlen + d->block - 1) / d->block) return 0;
        return chunk_layout(d).total;
    }
    if (d->route == BDGDN_ROUTE_SPLIT) {
        if (!split_supported(ty, d->d_k, d->d_v, lp_of(d->block))) return 0;
        return (size_t)total_blocks(d) * d->h_v * d->d_k * d->d_v * sizeof(float);   // seed states
    }
    if (d->route != BDGDN_ROUTE_FUSED && d->route != BDGDN_ROUTE_RECORDS) return 0;
    if (one_kernel(d, ty)) return 0;
    return (size_t)total_blocks(d) * d->h_v * scan_record_bytes(ty, lp_of(d->block));
}

size_t bdgdn_fwd_train_workspace(const bdgdn_fwd_desc_t *desc)
{
    if (!desc) return 0;
    // size only descriptors whose shapes and types are valid (packing is checked per call)
    if (check_heads(desc->h_qk, desc->h_v, desc->d_k, desc->d_v, desc->block, desc->scale, desc->dtype,
                    desc->out_dtype) != BDGDN_OK)
        return 0;
    if (desc->batch <= 0 || desc->seqlen < 0) return 0;
    return workspace_bytes_of(desc);
}

int bdgdn_fwd_train(const bdgdn_fwd_desc_t *desc, const void *q, const void *k, const void *v,
                    const float *g, const float *beta, const void *qn, const void *kn,
                    const void *vn, const float *gn, const float *betan,
                    const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                    const float *h0, void *o, void *on, float *ht, void *workspace,
                    size_t workspace_bytes, void *stream)
{
    int st = check_fwd(desc, cu_seqlens_dev, cu_seqlens_host);
    if (st != BDGDN_OK) return st;
    if (!q || !k || !v || !g || !beta || !qn || !kn || !vn || !gn || !betan || !o || !on)
        return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(qn) || !aligned16(kn) ||
        !aligned16(vn) || !aligned16(o) || !aligned16(on))
        return BDGDN_ERR_INVALID_ARG;
    const size_t need = workspace_bytes_of(desc);
    if (need > 0 && (workspace_bytes < need || !workspace)) return BDGDN_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return BDGDN_ERR_WORKSPACE;
    const bool packed = desc->num_seqs > 0;
    const int nseq = packed ? desc->num_seqs : desc->batch;
    if (desc->seqlen == 0) return BDGDN_OK;
    Types ty;
    types_of(desc->dtype, desc->out_dtype, ty);
    const int lp = lp_of(desc->block);
    const hipStream_t strm = static_cast<hipStream_t>(stream);
    // longest documents first, so that the longest serial chains start first
    int order[kMaxOrder];
    int n_order = 0;
    if (packed && nseq <= kMaxOrder) {
        std::vector<int> idx(nseq);
        std::iota(idx.begin(), idx.end(), 0);
        std::stable_sort(idx.begin(), idx.end(), [&](int x, int y) {
            return cu_seqlens_host[x + 1] - cu_seqlens_host[x] > cu_seqlens_host[y + 1] - cu_seqlens_host[y];
        });
        for (int i = 0; i < nseq; ++i) order[i] = idx[i];
        n_order = nseq;
    }
    hipError_t e;
    const bool wide = desc->route == BDGDN_ROUTE_FUSED && fused_uses_wide_pass(desc, ty);
    if (desc->route == BDGDN_ROUTE_CHUNKED || wide) {
        ChunkArgs ca = {};
        ca.q = q; ca.k = k; ca.v = v; ca.qn = qn; ca.kn = kn; ca.vn = vn;
        ca.g = g; ca.beta = beta; ca.gn = gn; ca.betan = betan;
        ca.cu = packed ? cu_seqlens_dev : nullptr;
        ca.h0 = h0; ca.ht = ht; ca.o = o; ca.on = on;
        const ChunkLayout lay = chunk_layout(desc);
        ca.rec = static_cast<unsigned char *>(workspace) + lay.rec;
        ca.ckpt = reinterpret_cast<float *>(static_cast<unsigned char *>(workspace) + lay.ckpt);
        ca.T = desc->seqlen; ca.L = desc->block; ca.nblk = (desc->seqlen + desc->block - 1) / desc->block;
        ca.h_qk = desc->h_qk; ca.h_v = desc->h_v; ca.dv = desc->d_v;
        // the fused route's wide pass: every chain one segment, all d_v columns together
        const ChunkPlan plan = wide ? ChunkPlan{1, std::max(16, ca.nblk)} : chunk_plan(desc);
        const int G = plan.G;
        ca.G = G;
        ca.n_ot = plan.tiles;
        auto nseg = [&](long len) {   // an empty document is one segment without blocks (it writes ht)
            const long nb = (len + desc->block - 1) / desc->block;
            return nb <= 0 ? 1 : (int)((nb + G - 1) / G);
        };
        long segs = 0;
        int n1 = 0, max_seg = 1;
        if (packed) {
            for (int i = 0; i < nseq; ++i) {
                const int doc = order[i];
                const int ns = nseg(cu_seqlens_host[doc + 1] - cu_seqlens_host[doc]);
                if (segs >= (1L << 21)) return BDGDN_ERR_UNSUPPORTED;
                ca.order[i] = doc | (int)(segs << 10);
                segs += ns;
                if (ns >= 2) ++n1;
                max_seg = std::max(max_seg, ns);
            }
            ca.n_order = nseq;
        } else {
            const int ns = nseg(desc->seqlen);
            segs = (long)ns * nseq;
            n1 = ns >= 2 ? nseq : 0;
            max_seg = ns;
            ca.n_order = 0;
        }
        ca.n1 = n1;
        ca.J_max = (max_seg - 1) * G;
        ca.n_groups = (int)(segs * desc->h_qk);
        ca.n_vt = desc->d_v / 32;
        ca.scale = desc->scale;
        e = launch_fwd_chunked(ty, desc->d_k, lp, ca, strm);
        return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
    }
    if (desc->route != BDGDN_ROUTE_ONEPASS) {
        IntraArgs ia;
        ia.q = q; ia.k = k; ia.qn = qn; ia.kn = kn;
        ia.g = g; ia.beta = beta; ia.gn = gn; ia.betan = betan;
        ia.ws = static_cast<unsigned char *>(workspace);
        ia.T = desc->seqlen; ia.L = desc->block;
        ia.nblk = (desc->seqlen + desc->block - 1) / desc->block;
        ia.total_blocks = total_blocks(desc);
        ia.h_qk = desc->h_qk; ia.h_v = desc->h_v;
        ScanArgs sa = {};
        sa.q = q; sa.k = k; sa.v = v; sa.qn = qn; sa.kn = kn; sa.vn = vn;
        sa.g = g; sa.beta = beta; sa.gn = gn; sa.betan = betan;
        sa.cu = packed ? cu_seqlens_dev : nullptr;
        sa.h0 = h0; sa.ht = ht; sa.o = o; sa.on = on;
        sa.ws = static_cast<const unsigned char *>(workspace);
        sa.bs = desc->route == BDGDN_ROUTE_SPLIT ? static_cast<float *>(workspace) : nullptr;
        sa.T = desc->seqlen; sa.L = desc->block; sa.nblk = ia.nblk;
        sa.h_qk = desc->h_qk; sa.h_v = desc->h_v; sa.dv = desc->d_v;
        sa.n_chains = nseq * desc->h_v;
        sa.n_vt = desc->d_v / scan_tile_v();
        sa.scale = desc->scale;
        sa.n_order = n_order;
        for (int i = 0; i < n_order; ++i) sa.order[i] = order[i];
        if (desc->route == BDGDN_ROUTE_SPLIT) {
            NoisyArgs na;
            na.qn = qn; na.kn = kn; na.vn = vn; na.gn = gn; na.betan = betan;
            na.bs = static_cast<const float *>(sa.bs);
            na.cu = sa.cu;
            na.on = on;
            na.T = desc->seqlen; na.L = desc->block; na.nblk = ia.nblk;
            na.n_docs = packed ? nseq : 0;
            na.total_blocks = ia.total_blocks;
            na.h_qk = desc->h_qk; na.h_v = desc->h_v;
            na.scale = desc->scale;
            e = launch_fwd_split(ty, lp, sa, na, strm);
        } else {
            e = one_kernel(desc, ty) ? launch_one_kernel(desc, ty, sa, strm)
                                     : launch_fwd_scan(ty, desc->d_k, lp, ia, sa, strm);
        }
    } else {
        FwdArgs a;
        a.q = q; a.k = k; a.v = v; a.qn = qn; a.kn = kn; a.vn = vn;
        a.g = g; a.beta = beta; a.gn = gn; a.betan = betan;
        a.cu = packed ? cu_seqlens_dev : nullptr;
        a.h0 = h0; a.ht = ht; a.o = o; a.on = on;
        a.T = desc->seqlen; a.h_qk = desc->h_qk; a.h_v = desc->h_v; a.dv = desc->d_v; a.L = desc->block;
        a.n_chains = nseq * desc->h_v;
        a.n_vt = desc->d_v / fwd_tile_v();
        a.scale = desc->scale;
        a.n_order = n_order;
        for (int i = 0; i < n_order; ++i) a.order[i] = order[i];
        e = launch_fwd_fused(ty, desc->d_k, lp, a, strm);
    }
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

static int check_serve(const bdgdn_serve_desc_t *d)
{
    if (!d) return BDGDN_ERR_INVALID_ARG;
    if (d->num_req < 0) return BDGDN_ERR_INVALID_ARG;
    return check_heads(d->h_qk, d->h_v, d->d_k, d->d_v, d->block, d->scale, d->dtype, d->out_dtype);
}

static ServeArgs serve_args(const bdgdn_serve_desc_t *d, const float *pool, const int32_t *slot,
                            const void *q, const void *k, const void *v, const float *g,
                            const float *beta, void *o)
{
    ServeArgs a;
    a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta;
    a.pool = const_cast<float *>(pool);
    a.slot = slot; a.o = o;
    a.R = d->num_req; a.h_qk = d->h_qk; a.h_v = d->h_v; a.dv = d->d_v; a.L = d->block;
    a.n_vt = d->d_v / serve_tile_v();
    a.scale = d->scale;
    a.states = nullptr;
    a.n_rec = 0;
    a.accept = nullptr;
    return a;
}

int bdgdn_denoise_step(const bdgdn_serve_desc_t *desc, const float *state_pool,
                       const int32_t *slot, const void *q, const void *k, const void *v,
                       const float *g, const float *beta, void *o, void *stream)
{
    int st = check_serve(desc);
    if (st != BDGDN_OK) return st;
    if (!state_pool || !q || !k || !v || !g || !beta || !o) return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return BDGDN_ERR_INVALID_ARG;
    if (desc->num_req == 0) return BDGDN_OK;
    ServeArgs a = serve_args(desc, state_pool, slot, q, k, v, g, beta, o);
    Types ty;
    types_of(desc->dtype, desc->out_dtype, ty);
    hipError_t e = launch_denoise(ty, desc->d_k, lp_of(desc->block), a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

int bdgdn_commit(const bdgdn_serve_desc_t *desc, float *state_pool, const int32_t *slot,
                 const void *q, const void *k, const void *v, const float *g,
                 const float *beta, void *o_causal, void *stream)
{
    int st = check_serve(desc);
    if (st != BDGDN_OK) return st;
    if (!state_pool || !q || !k || !v || !g || !beta) return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o_causal)) return BDGDN_ERR_INVALID_ARG;
    if (desc->num_req == 0) return BDGDN_OK;
    ServeArgs a = serve_args(desc, state_pool, slot, q, k, v, g, beta, o_causal);
    Types ty;
    types_of(desc->dtype, desc->out_dtype, ty);
    hipError_t e = launch_commit(ty, desc->d_k, lp_of(desc->block), o_causal != nullptr, a,
                                 static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

int bdgdn_commit_record(const bdgdn_serve_desc_t *desc, float *state_pool, const int32_t *slot,
                        const void *q, const void *k, const void *v, const float *g,
                        const float *beta, void *o_causal, int32_t n_record, float *states,
                        void *stream)
{
    int st = check_serve(desc);
    if (st != BDGDN_OK) return st;
    if (!state_pool || !q || !k || !v || !g || !beta || !states) return BDGDN_ERR_INVALID_ARG;
    if (n_record < 1 || n_record > desc->block) return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o_causal) || !aligned16(states))
        return BDGDN_ERR_INVALID_ARG;
    Types ty;
    types_of(desc->dtype, desc->out_dtype, ty);
    if (!record_supported(ty, desc->d_k, desc->d_v, lp_of(desc->block))) return BDGDN_ERR_UNSUPPORTED;
    if (desc->num_req == 0) return BDGDN_OK;
    ServeArgs a = serve_args(desc, state_pool, slot, q, k, v, g, beta, o_causal);
    a.states = states;
    a.n_rec = n_record;
    hipError_t e = launch_commit_record(ty, lp_of(desc->block), o_causal != nullptr, a,
                                        static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

int bdgdn_accept_states(const bdgdn_serve_desc_t *desc, float *state_pool, const int32_t *slot,
                        const float *states, int32_t n_record, const int32_t *accept, void *stream)
{
    int st = check_serve(desc);
    if (st != BDGDN_OK) return st;
    if (!state_pool || !states || !accept) return BDGDN_ERR_INVALID_ARG;
    if (n_record < 1 || n_record > desc->block) return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(state_pool) || !aligned16(states)) return BDGDN_ERR_INVALID_ARG;
    if (desc->num_req == 0) return BDGDN_OK;
    ServeArgs a = serve_args(desc, state_pool, slot, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    a.states = const_cast<float *>(states);
    a.n_rec = n_record;
    a.accept = accept;
    hipError_t e = launch_accept_states(a, desc->d_k, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

// The views forward: FUSED runs the one-kernel forward once per view (any block it takes);
// SPLIT writes the seeds in the one-kernel forward and needs blocks of at most 32.
static bool views_supported(const bdgdn_fwd_desc_t *d)
{
    Types ty;
    if (!types_of(d->dtype, d->out_dtype, ty)) return false;
    if (d->route == BDGDN_ROUTE_SPLIT)
        return split_supported(ty, d->d_k, d->d_v, lp_of(d->block)) && pipelined_supported(ty, d->d_k, lp_of(d->block));
    return pipelined_supported(ty, d->d_k, lp_of(d->block)) || pair_blocks(d, ty);
}

size_t bdgdn_fwd_train_views_workspace(const bdgdn_fwd_desc_t *desc)
{
    if (!desc || check_heads(desc->h_qk, desc->h_v, desc->d_k, desc->d_v, desc->block, desc->scale, desc->dtype,
                             desc->out_dtype) != BDGDN_OK)
        return 0;
    if (desc->batch <= 0 || desc->seqlen <= 0 || !views_supported(desc)) return 0;
    if (desc->route != BDGDN_ROUTE_SPLIT) return 0;   // the fused schedule needs no workspace
    // the seeds (needed from the second view on; sized for any number of views)
    return (size_t)total_blocks(desc) * desc->h_v * desc->d_k * desc->d_v * sizeof(float);
}

int bdgdn_fwd_train_views(const bdgdn_fwd_desc_t *desc, const void *q, const void *k, const void *v,
                          const float *g, const float *beta, const bdgdn_noisy_view_t *views, int32_t n_views,
                          const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host, const float *h0,
                          void *o, float *ht, void *workspace, size_t workspace_bytes, void *stream)
{
    int st = check_fwd(desc, cu_seqlens_dev, cu_seqlens_host);
    if (st != BDGDN_OK) return st;
    if (!views_supported(desc)) return BDGDN_ERR_UNSUPPORTED;
    if (desc->route != BDGDN_ROUTE_FUSED && desc->route != BDGDN_ROUTE_SPLIT) return BDGDN_ERR_UNSUPPORTED;
    if (!q || !k || !v || !g || !beta || !o || !views || n_views < 1 || n_views > 16) return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return BDGDN_ERR_INVALID_ARG;
    for (int i = 0; i < n_views; ++i) {
        const bdgdn_noisy_view_t &w = views[i];
        if (!w.q || !w.k || !w.v || !w.g || !w.beta || !w.o) return BDGDN_ERR_INVALID_ARG;
        if (!aligned16(w.q) || !aligned16(w.k) || !aligned16(w.v) || !aligned16(w.o)) return BDGDN_ERR_INVALID_ARG;
    }
    if (desc->seqlen == 0) return BDGDN_OK;
    const bool split = desc->route == BDGDN_ROUTE_SPLIT && n_views > 1;
    const size_t need = split ? bdgdn_fwd_train_views_workspace(desc) : 0;
    if (need > 0 && (workspace_bytes < need || !workspace)) return BDGDN_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return BDGDN_ERR_WORKSPACE;
    const bool packed = desc->num_seqs > 0;
    const int nseq = packed ? desc->num_seqs : desc->batch;
    const hipStream_t strm = static_cast<hipStream_t>(stream);
    const int lp = lp_of(desc->block);
    const bool f32_out = desc->out_dtype == BDGDN_F32;
    ScanArgs sa = {};
    sa.q = q; sa.k = k; sa.v = v;
    sa.qn = views[0].q; sa.kn = views[0].k; sa.vn = views[0].v;
    sa.g = g; sa.beta = beta; sa.gn = views[0].g; sa.betan = views[0].beta;
    sa.cu = packed ? cu_seqlens_dev : nullptr;
    sa.h0 = h0; sa.ht = ht; sa.o = o; sa.on = nullptr;
    sa.ws = nullptr;
    sa.bs = static_cast<float *>(workspace);
    sa.T = desc->seqlen; sa.L = desc->block; sa.nblk = (desc->seqlen + desc->block - 1) / desc->block;
    sa.h_qk = desc->h_qk; sa.h_v = desc->h_v; sa.dv = desc->d_v;
    sa.n_chains = nseq * desc->h_v;
    sa.n_vt = desc->d_v / scan_tile_v();
    sa.scale = desc->scale;
    sa.n_order = 0;
    if (packed && nseq <= kMaxOrder) {
        std::vector<int> idx(nseq);
        std::iota(idx.begin(), idx.end(), 0);
        std::stable_sort(idx.begin(), idx.end(), [&](int x, int y) {
            return cu_seqlens_host[x + 1] - cu_seqlens_host[x] > cu_seqlens_host[y + 1] - cu_seqlens_host[y];
        });
        for (int i = 0; i < nseq; ++i) sa.order[i] = idx[i];
        sa.n_order = nseq;
    }
    Types ty;
    types_of(desc->dtype, desc->out_dtype, ty);
    hipError_t e;
    if (!split) {
        // FUSED: one on-chip pass per view (the clean scan recomputed with each; its outputs
        // and ht written by the first only)
        sa.bs = nullptr;
        for (int i = 0; i < n_views; ++i) {
            sa.qn = views[i].q; sa.kn = views[i].k; sa.vn = views[i].v;
            sa.gn = views[i].g; sa.betan = views[i].beta;
            sa.on = views[i].o;
            sa.ht = i == 0 ? ht : nullptr;
            e = launch_one_kernel(desc, ty, sa, strm, i == 0);
            if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
        }
        return BDGDN_OK;
    }
    // SPLIT: view 0 in the one-kernel forward, which also writes the seed of every
    // (block, v-head); every further view from the seeds
    sa.on = views[0].o;
    e = launch_fwd_pipelined_seeds(ty, lp, sa, strm);
    if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
    for (int i = 1; i < n_views; ++i) {
        NoisyArgs na = {};
        na.qn = views[i].q; na.kn = views[i].k; na.vn = views[i].v;
        na.gn = views[i].g; na.betan = views[i].beta;
        na.bs = static_cast<const float *>(sa.bs);
        na.cu = sa.cu;
        na.on = views[i].o;
        na.T = desc->seqlen; na.L = desc->block; na.nblk = sa.nblk;
        na.n_docs = packed ? nseq : 0;
        na.total_blocks = total_blocks(desc);
        na.h_qk = desc->h_qk; na.h_v = desc->h_v;
        na.scale = desc->scale;
        e = launch_noisy_blocks(lp, f32_out, na, strm);
        if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
    }
    return BDGDN_OK;
}

// The block-form backward: bf16 inputs, d_k = d_v = 128, blocks of at most 32 positions, or
// of an even 34 .. 64 (noisy blocks of two sub-blocks, the clean stream in sub-blocks of half
// the block).
static bool bwd_shape_ok(const bdgdn_fwd_desc_t *d)
{
    return d->dtype == BDGDN_BF16 && d->d_k == 128 && d->d_v == 128 &&
           (d->block <= 32 || (d->block <= 64 && d->block % 2 == 0));
}
static bool bwd_pairs(const bdgdn_fwd_desc_t *d) { return d->block > 32; }
// The clean block of the block-form backward: the block, or half of it for pairs.
static bdgdn_fwd_desc_t bwd_sub(const bdgdn_fwd_desc_t *d)
{
    bdgdn_fwd_desc_t s = *d;
    if (bwd_pairs(d)) s.block = d->block / 2;
    return s;
}

// Workspace of the backward, per (global block, v-head): the seed state (fp16), the part of
// the state gradient at the block's start that does not depend on dh (fp16, tile-native;
// the reverse scan overwrites it with dh at the block's end, which the clean block kernel
// uses as fp16 operands only), U K (32 x d_k, fp16), gamma_n (fp32); then the range pass's
// per-block maxima and {sigma, 1 / sigma}.  Byte offsets, each aligned to 256.
struct BwdLayout {
    size_t seeds, cterm, uk, gnb, part, range, total;
};
static size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }
static BwdLayout bwd_layout_units(size_t units, const bdgdn_fwd_desc_t *d, size_t base)
{
    const size_t st = (size_t)d->d_k * d->d_v;
    BwdLayout l;
    l.seeds = base;
    l.cterm = l.seeds + up256(units * st * 2);
    l.uk = l.cterm + up256(units * st * 2);
    l.gnb = l.uk + up256(units * 32 * d->d_k * 2);
    l.part = l.gnb + up256(units * 4);
    l.range = l.part + up256(kRangeBlocks * 4);
    l.total = l.range + 256;
    return l;
}
static BwdLayout bwd_layout(const bdgdn_fwd_desc_t *d)
{
    const bdgdn_fwd_desc_t sub = bwd_sub(d);
    return bwd_layout_units((size_t)total_blocks(&sub) * d->h_v, d, 0);
}

// The time-segmented block-form backward (Appendix "Backward primitives", the strided clean
// checkpoints of the checkpoint build and "Choosing the stride"): every chain's clean blocks
// (sub-blocks for noisy blocks of two) cut into segments of seg_len, the clean state kept
// at each segment start after the first (fp32, one per chain), the segments then run last
// first, each recomputing its own seeds from its checkpoint, so that the per-block
// workspace holds one segment.  Segment 0 holds the most blocks: every chain contributes
// min(its blocks, seg_len) to it.
struct SegPlan {
    int n_seg = 1, seg_len = 0;
    long max_units = 0;               // clean (sub-)blocks of segment 0, all sequences
    std::vector<long> units, pairs;   // per segment: clean (sub-)blocks, noisy blocks of two
};
static long chain_blocks(const bdgdn_fwd_desc_t *d, const int32_t *cu_host, int n, int Lc)
{
    const long len = d->num_seqs > 0 ? (long)cu_host[n + 1] - cu_host[n] : d->seqlen;
    return (len + Lc - 1) / Lc;
}
// The plan for `segments` segments (fewer when the chains are short); false when packed
// lengths are missing or invalid.  With counts = false only n_seg, seg_len and max_units.
static bool seg_plan(const bdgdn_fwd_desc_t *d, const int32_t *cu_host, int segments, bool counts, SegPlan &p)
{
    const bool packed = d->num_seqs > 0;
    const int nseq = packed ? d->num_seqs : d->batch;
    if (segments < 1 || (packed && !cu_host)) return false;
    if (packed && (cu_host[0] != 0 || cu_host[nseq] != d->seqlen)) return false;
    const int Lc = bwd_sub(d).block;
    long maxnb = 0;
    for (int n = 0; n < nseq; ++n) {
        if (packed && cu_host[n + 1] < cu_host[n]) return false;
        maxnb = std::max(maxnb, chain_blocks(d, cu_host, n, Lc));
    }
    if (maxnb == 0) return false;
    long S = (maxnb + segments - 1) / segments;
    if (bwd_pairs(d)) S += S & 1;   // segments start on noisy-block boundaries
    p.seg_len = (int)S;
    p.n_seg = (int)((maxnb + S - 1) / S);
    p.max_units = 0;
    for (int n = 0; n < nseq; ++n) p.max_units += std::min(chain_blocks(d, cu_host, n, Lc), S);
    if (counts) {
        p.units.assign(p.n_seg, 0);
        p.pairs.assign(p.n_seg, 0);
        for (int n = 0; n < nseq; ++n) {
            const long nb = chain_blocks(d, cu_host, n, Lc);
            for (int k = 0; k < p.n_seg; ++k) {
                const long c = std::max(0L, std::min(nb - (long)k * S, S));
                p.units[k] += c;
                p.pairs[k] += (c + 1) / 2;
            }
        }
    }
    return true;
}
// Workspace of the segmented backward: the checkpoints at segment starts 1 .. n_seg - 1, the
// state-gradient carry (fp32 [seq][h_v][d_k][d_v] each), the segment tables, then the
// per-block layout for segment 0's blocks.
struct SegLayout {
    size_t ckpt, carry, tab;
    BwdLayout body;
};
static SegLayout seg_layout(const bdgdn_fwd_desc_t *d, const SegPlan &p)
{
    const int nseq = d->num_seqs > 0 ? d->num_seqs : d->batch;
    const size_t state = (size_t)nseq * d->h_v * d->d_k * d->d_v * sizeof(float);
    SegLayout l;
    l.ckpt = 0;
    l.carry = l.ckpt + up256((size_t)(p.n_seg - 1) * state);
    l.tab = l.carry + up256(state);
    const size_t tab_bytes = 2 * (size_t)p.n_seg * (nseq + 1) * sizeof(int);
    l.body = bwd_layout_units((size_t)p.max_units * d->h_v, d, l.tab + up256(tab_bytes));
    return l;
}

// Shapes outside the block-form kernels run the per-step fp32 backward (bwd_generic.hip).
static bool bwd_generic_ok(const bdgdn_fwd_desc_t *d, int n_views)
{
    return !bwd_shape_ok(d) && d->num_seqs <= kMaxOrder &&
           bwd_generic_supported(d->dtype == BDGDN_F32, d->d_k, d->d_v, d->block, n_views);
}
static size_t bwd_generic_bytes(const bdgdn_fwd_desc_t *d)
{
    const int nseq = d->num_seqs > 0 ? d->num_seqs : d->batch;
    return bwd_generic_workspace(nseq, total_blocks(d), d->h_v, d->d_k, d->d_v);
}

size_t bdgdn_bwd_train_workspace(const bdgdn_fwd_desc_t *desc)
{
    if (!desc || check_heads(desc->h_qk, desc->h_v, desc->d_k, desc->d_v, desc->block, desc->scale, desc->dtype,
                             desc->out_dtype) != BDGDN_OK)
        return 0;
    if (desc->batch <= 0 || desc->seqlen <= 0) return 0;
    if (bwd_shape_ok(desc)) return bwd_layout(desc).total;
    return bwd_generic_ok(desc, 1) ? bwd_generic_bytes(desc) : 0;
}

size_t bdgdn_bwd_train_workspace_segmented(const bdgdn_fwd_desc_t *desc, const int32_t *cu_seqlens_host,
                                           int segments)
{
    const size_t full = bdgdn_bwd_train_workspace(desc);
    if (full == 0 || segments < 1) return 0;
    if (!bwd_shape_ok(desc) || segments == 1) return full;
    SegPlan p;
    if (!seg_plan(desc, cu_seqlens_host, segments, false, p)) return 0;
    return p.n_seg > 1 ? seg_layout(desc, p).body.total : full;
}

// The backward of the clean stream and noisy view 0 (qn .. dbetan), plus n_more further views.
static int bwd_impl(const bdgdn_fwd_desc_t *desc, const void *q, const void *k, const void *v, const float *g,
                    const float *beta, const void *qn, const void *kn, const void *vn, const float *gn,
                    const float *betan, const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                    const float *h0, const void *dout, const void *doutn, const float *dht, float *dq, float *dk,
                    float *dv, float *dg, float *dbeta, float *dqn, float *dkn, float *dvn, float *dgn,
                    float *dbetan, float *dh0, const BwdView *more, int n_more, void *workspace,
                    size_t workspace_bytes, void *stream)
{
    int st = check_fwd(desc, cu_seqlens_dev, cu_seqlens_host);
    if (st != BDGDN_OK) return st;
    const bool generic = !bwd_shape_ok(desc);
    if (generic && !bwd_generic_ok(desc, 1 + n_more)) return BDGDN_ERR_UNSUPPORTED;
    if (!q || !k || !v || !g || !beta || !qn || !kn || !vn || !gn || !betan || !dout || !doutn || !dq ||
        !dk || !dv || !dg || !dbeta || !dqn || !dkn || !dvn || !dgn || !dbetan)
        return BDGDN_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(qn) || !aligned16(kn) ||
        !aligned16(vn) || !aligned16(dout) || !aligned16(doutn) || !aligned16(h0) || !aligned16(dht))
        return BDGDN_ERR_INVALID_ARG;
    for (int i = 0; i < n_more; ++i) {
        const BwdView &w = more[i];
        if (!w.q || !w.k || !w.v || !w.g || !w.beta || !w.dout || !w.dq || !w.dk || !w.dv || !w.dg || !w.db)
            return BDGDN_ERR_INVALID_ARG;
        if (!aligned16(w.q) || !aligned16(w.k) || !aligned16(w.v) || !aligned16(w.dout)) return BDGDN_ERR_INVALID_ARG;
    }
    if (desc->seqlen == 0) return BDGDN_OK;
    const size_t need = bdgdn_bwd_train_workspace(desc);
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return BDGDN_ERR_WORKSPACE;
    // below the full workspace, the block-form backward runs in the fewest time segments
    // whose workspace fits
    SegPlan plan;
    bool segmented = false;
    if (workspace_bytes < need) {
        if (generic) return BDGDN_ERR_WORKSPACE;
        int K = 2;
        for (;; ++K) {
            if (!seg_plan(desc, cu_seqlens_host, K, false, plan)) return BDGDN_ERR_WORKSPACE;
            if (plan.n_seg > 1 && seg_layout(desc, plan).body.total <= workspace_bytes) break;
            if (plan.seg_len <= (bwd_pairs(desc) ? 2 : 1)) return BDGDN_ERR_WORKSPACE;   // no finer segments
        }
        seg_plan(desc, cu_seqlens_host, K, true, plan);
        segmented = true;
    }
    const bool packed = desc->num_seqs > 0;
    const int nseq = packed ? desc->num_seqs : desc->batch;
    const hipStream_t strm = static_cast<hipStream_t>(stream);
    if (generic) {
        GenBwdCall c = {};
        c.q = q; c.k = k; c.v = v; c.g = g; c.beta = beta; c.dout = dout;
        c.dq = dq; c.dk = dk; c.dv = dv; c.dg = dg; c.db = dbeta;
        c.qn = qn; c.kn = kn; c.vn = vn; c.gn = gn; c.betan = betan; c.doutn = doutn;
        c.dqn = dqn; c.dkn = dkn; c.dvn = dvn; c.dgn = dgn; c.dbn = dbetan;
        c.more = more; c.n_more = n_more;
        c.cu = packed ? cu_seqlens_dev : nullptr;
        c.cu_host = packed ? cu_seqlens_host : nullptr;
        c.n_seq = nseq;
        c.rows = (long)desc->batch * desc->seqlen;
        c.total_blocks = total_blocks(desc);
        c.h0 = h0; c.dht = dht; c.dh0 = dh0;
        c.T = desc->seqlen; c.L = desc->block; c.h_qk = desc->h_qk; c.h_v = desc->h_v;
        c.d_k = desc->d_k; c.d_v = desc->d_v;
        c.scale = desc->scale;
        c.workspace = workspace;
        const hipError_t e = launch_bwd_generic(desc->dtype == BDGDN_F32, desc->out_dtype == BDGDN_F32, c, strm);
        return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
    }
    unsigned char *ws = static_cast<unsigned char *>(workspace);
    const SegLayout sl = segmented ? seg_layout(desc, plan) : SegLayout{};
    const BwdLayout lay = segmented ? sl.body : bwd_layout(desc);
    _Float16 *seeds = reinterpret_cast<_Float16 *>(ws + lay.seeds);
    const bdgdn_fwd_desc_t sub = bwd_sub(desc);   // the clean blocks
    const int Lc = sub.block;
    // 1. the clean scan from h0, writing the seed state of every block (fp16: the block
    // kernels stage it as fp16 MFMA operands)
    ScanArgs sa = {};
    sa.q = q; sa.k = k; sa.v = v; sa.qn = qn; sa.kn = kn; sa.vn = vn;
    sa.g = g; sa.beta = beta; sa.gn = gn; sa.betan = betan;
    sa.cu = packed ? cu_seqlens_dev : nullptr;
    sa.h0 = h0; sa.ht = nullptr;
    sa.o = ws; sa.on = nullptr;   // never written: the states-only scan has no outputs
    sa.ws = nullptr;
    sa.bs = seeds;
    sa.T = desc->seqlen; sa.L = Lc; sa.nblk = (desc->seqlen + Lc - 1) / Lc;
    sa.h_qk = desc->h_qk; sa.h_v = desc->h_v; sa.dv = desc->d_v;
    sa.n_chains = nseq * desc->h_v;
    sa.n_vt = desc->d_v / scan_tile_v();
    sa.scale = desc->scale;
    sa.n_order = 0;
    if (packed && nseq <= kMaxOrder) {
        std::vector<int> idx(nseq);
        std::iota(idx.begin(), idx.end(), 0);
        std::stable_sort(idx.begin(), idx.end(), [&](int x, int y) {
            return cu_seqlens_host[x + 1] - cu_seqlens_host[x] > cu_seqlens_host[y + 1] - cu_seqlens_host[y];
        });
        for (int i = 0; i < nseq; ++i) sa.order[i] = idx[i];
        sa.n_order = nseq;
    }
    hipError_t e = hipSuccess;
    if (!segmented) {
        e = launch_scan_states(lp_of(Lc), false, true, sa, strm);
        if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
    }
    // 2. the reverse walk over the blocks of every (sequence, v-head)
    BwdArgs a = {};
    a.q = q; a.k = k; a.v = v; a.qn = qn; a.kn = kn; a.vn = vn;
    a.g = g; a.beta = beta; a.gn = gn; a.betan = betan;
    a.dout = dout; a.doutn = doutn;
    a.seeds = seeds; a.dht = dht;
    a.dq = dq; a.dk = dk; a.dv = dv; a.dg = dg; a.db = dbeta;
    a.dqn = dqn; a.dkn = dkn; a.dvn = dvn; a.dgn = dgn; a.dbn = dbetan;
    a.dh0 = dh0;
    a.cterm = reinterpret_cast<_Float16 *>(ws + lay.cterm);
    a.dh = a.cterm;   // the scan writes dh_b over cterm_b once it has read it
    a.uk = reinterpret_cast<_Float16 *>(ws + lay.uk);
    a.gnb = reinterpret_cast<float *>(ws + lay.gnb);
    a.cu = sa.cu;
    a.n_docs = packed ? nseq : 0;
    a.n_chains = nseq * desc->h_v;
    a.T = desc->seqlen; a.nblk = sa.nblk; a.L = Lc;
    a.h_qk = desc->h_qk; a.h_v = desc->h_v;
    a.scale = desc->scale;
    const long rows = (long)desc->batch * desc->seqlen;
    // the range of the upstream gradients: the power-of-two scale they enter the kernels with
    RangeArgs ra = {};
    ra.arr[ra.count] = dout; ra.n[ra.count++] = rows * desc->h_v * desc->d_v;
    ra.arr[ra.count] = doutn; ra.n[ra.count++] = rows * desc->h_v * desc->d_v;
    for (int i = 0; i < n_more; ++i) {
        ra.arr[ra.count] = more[i].dout;
        ra.n[ra.count++] = rows * desc->h_v * desc->d_v;
    }
    if (dht) {
        ra.arr[ra.count] = dht;
        ra.n[ra.count++] = (long)nseq * desc->h_v * desc->d_k * desc->d_v;
        ra.last_f32 = true;
    }
    ra.part = reinterpret_cast<float *>(ws + lay.part);
    ra.range = reinterpret_cast<float *>(ws + lay.range);
    a.range = ra.range;
    e = launch_bwd_range(desc->out_dtype == BDGDN_BF16, ra, strm);
    if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
    if (!segmented) {
        e = launch_bwd(desc->out_dtype == BDGDN_BF16, a, more, n_more, nseq * desc->h_v,
                       total_blocks(&sub) * desc->h_v, bwd_pairs(desc) ? total_blocks(desc) * desc->h_v : 0, strm);
        return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
    }
    // time segments: the tables, the checkpoints by a forward pass over segments 0 ..
    // n_seg - 2, then each segment last first: its seeds from its checkpoint, its blocks
    const size_t state = (size_t)nseq * desc->h_v * desc->d_k * desc->d_v;
    float *ckpt = reinterpret_cast<float *>(ws + sl.ckpt);   // segment k's start state at ckpt + (k - 1) state
    int *tab = reinterpret_cast<int *>(ws + sl.tab), *tabp = tab + (size_t)plan.n_seg * (nseq + 1);
    e = launch_bwd_seg_plan(packed ? cu_seqlens_dev : nullptr, nseq, desc->seqlen, Lc, plan.seg_len, plan.n_seg, tab,
                            tabp, strm);
    if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
    auto seg_states = [&](int k, bool checkpoint) {
        sa.seg = tab + (size_t)k * (nseq + 1);
        sa.blk0 = k * plan.seg_len;
        sa.seg_len = plan.seg_len;
        sa.h0 = k > 0 ? ckpt + (size_t)(k - 1) * state : h0;
        sa.ht = checkpoint ? ckpt + (size_t)k * state : nullptr;
        return launch_scan_states(lp_of(Lc), false, true, sa, strm);
    };
    for (int k = 0; k + 1 < plan.n_seg; ++k)
        if (seg_states(k, true) != hipSuccess) return BDGDN_ERR_LAUNCH;
    a.carry = reinterpret_cast<float *>(ws + sl.carry);
    a.seg_len = plan.seg_len;
    for (int k = plan.n_seg - 1; k >= 0; --k) {
        if (seg_states(k, false) != hipSuccess) return BDGDN_ERR_LAUNCH;
        a.seg = tab + (size_t)k * (nseq + 1);
        a.segp = tabp + (size_t)k * (nseq + 1);
        a.blk0 = k * plan.seg_len;
        e = launch_bwd(desc->out_dtype == BDGDN_BF16, a, more, n_more, nseq * desc->h_v, plan.units[k] * desc->h_v,
                       bwd_pairs(desc) ? plan.pairs[k] * desc->h_v : 0, strm);
        if (e != hipSuccess) return BDGDN_ERR_LAUNCH;
    }
    return BDGDN_OK;
}

int bdgdn_bwd_train(const bdgdn_fwd_desc_t *desc, const void *q, const void *k, const void *v,
                    const float *g, const float *beta, const void *qn, const void *kn,
                    const void *vn, const float *gn, const float *betan,
                    const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host, const float *h0,
                    const void *dout, const void *doutn, const float *dht,
                    float *dq, float *dk, float *dv, float *dg, float *dbeta,
                    float *dqn, float *dkn, float *dvn, float *dgn, float *dbetan, float *dh0,
                    void *workspace, size_t workspace_bytes, void *stream)
{
    return bwd_impl(desc, q, k, v, g, beta, qn, kn, vn, gn, betan, cu_seqlens_dev, cu_seqlens_host, h0, dout,
                    doutn, dht, dq, dk, dv, dg, dbeta, dqn, dkn, dvn, dgn, dbetan, dh0, nullptr, 0, workspace,
                    workspace_bytes, stream);
}

size_t bdgdn_bwd_train_views_workspace(const bdgdn_fwd_desc_t *desc) { return bdgdn_bwd_train_workspace(desc); }

int bdgdn_bwd_train_views(const bdgdn_fwd_desc_t *desc, const void *q, const void *k, const void *v,
                          const float *g, const float *beta, const bdgdn_noisy_view_grad_t *views, int32_t n_views,
                          const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host, const float *h0,
                          const void *dout, const float *dht, float *dq, float *dk, float *dv, float *dg,
                          float *dbeta, float *dh0, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!desc) return BDGDN_ERR_INVALID_ARG;
    if (!views || n_views < 1 || n_views > 16) return BDGDN_ERR_INVALID_ARG;
    BwdView more[16];
    for (int i = 1; i < n_views; ++i) {
        const bdgdn_noisy_view_grad_t &w = views[i];
        more[i - 1] = BwdView{w.q, w.k, w.v, w.g, w.beta, w.do_, w.dq, w.dk, w.dv, w.dg, w.dbeta};
    }
    const bdgdn_noisy_view_grad_t &w0 = views[0];
    return bwd_impl(desc, q, k, v, g, beta, w0.q, w0.k, w0.v, w0.g, w0.beta, cu_seqlens_dev, cu_seqlens_host, h0,
                    dout, w0.do_, dht, dq, dk, dv, dg, dbeta, w0.dq, w0.dk, w0.dv, w0.dg, w0.dbeta, dh0, more,
                    n_views - 1, workspace, workspace_bytes, stream);
}

size_t bdgdn_shortconv_bwd_workspace(const bdgdn_conv_desc_t *desc)
{
    if (!desc || desc->batch <= 0 || desc->seqlen < 0 || desc->channels <= 0 || desc->width < 1 || desc->width > 4)
        return 0;
    return conv_part_floats((long)desc->batch * desc->seqlen, desc->channels, desc->width) * sizeof(float);
}

int bdgdn_shortconv_fwd(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                        const float *bias, const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                        void *y, void *yn, void *stream)
{
    int st = check_conv(desc, cu_seqlens_dev, cu_seqlens_host);
    if (st != BDGDN_OK) return st;
    const bool any = (long)desc->batch * desc->seqlen > 0;   // token tensors may be NULL without rows
    if (!w || (any && (!x || !xn || !y || !yn))) return BDGDN_ERR_INVALID_ARG;
    if (!aligned8(x) || !aligned8(xn) || !aligned8(y) || !aligned8(yn)) return BDGDN_ERR_INVALID_ARG;
    const ConvArgs a = conv_args(desc, cu_seqlens_dev, x, xn, w, bias, y, yn);
    hipError_t e = launch_shortconv_fwd(desc->dtype == BDGDN_BF16, desc->width, a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

// Validation shared by the two ShortConv backward entry points.
static int check_conv_bwd(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                          const void *dy, const void *dyn, const int32_t *cu_seqlens_dev,
                          const int32_t *cu_seqlens_host, void *dx, void *dxn, float *dw)
{
    int st = check_conv(desc, cu_seqlens_dev, cu_seqlens_host);
    if (st != BDGDN_OK) return st;
    const bool any = (long)desc->batch * desc->seqlen > 0;
    if (!w || !dw || (any && (!x || !xn || !dy || !dyn || !dx || !dxn))) return BDGDN_ERR_INVALID_ARG;
    if (!aligned8(x) || !aligned8(xn) || !aligned8(dy) || !aligned8(dyn) || !aligned8(dx) || !aligned8(dxn))
        return BDGDN_ERR_INVALID_ARG;
    return BDGDN_OK;
}

static int conv_bwd_launch(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                           const float *bias, const void *dy, const void *dyn, const int32_t *cu_seqlens_dev,
                           void *dx, void *dxn, float *dw, float *dbias, float *part, hipStream_t stream)
{
    ConvArgs a = conv_args(desc, cu_seqlens_dev, x, xn, w, bias, dx, dxn);
    a.dy = dy; a.dyn = dyn;
    a.part = part;
    a.dw = dw;
    a.dbias = dbias;
    hipError_t e = launch_shortconv_bwd(desc->dtype == BDGDN_BF16, desc->width, a, stream);
    return e == hipSuccess ? BDGDN_OK : BDGDN_ERR_LAUNCH;
}

int bdgdn_shortconv_bwd(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                        const float *bias, const void *dy, const void *dyn, const int32_t *cu_seqlens_dev,
                        const int32_t *cu_seqlens_host, void *dx, void *dxn, float *dw, float *dbias,
                        void *workspace, size_t workspace_bytes, void *stream)
{
    int st = check_conv_bwd(desc, x, xn, w, dy, dyn, cu_seqlens_dev, cu_seqlens_host, dx, dxn, dw);
    if (st != BDGDN_OK) return st;
    const size_t need = bdgdn_shortconv_bwd_workspace(desc);
    if (need > 0 && (workspace_bytes < need || !workspace)) return BDGDN_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return BDGDN_ERR_WORKSPACE;
    return conv_bwd_launch(desc, x, xn, w, bias, dy, dyn, cu_seqlens_dev, dx, dxn, dw, dbias,
                           static_cast<float *>(workspace), static_cast<hipStream_t>(stream));
}

static_assert(BDGDN_NOALLOC_SCRATCH_BYTES == kConvScratchBytes, "the header states the scratch size");

int bdgdn_shortconv_bwd_noalloc(const bdgdn_conv_desc_t *desc, const void *x, const void *xn, const float *w,
                                const float *bias, const void *dy, const void *dyn, const int32_t *cu_seqlens_dev,
                                const int32_t *cu_seqlens_host, void *dx, void *dxn, float *dw, float *dbias,
                                void *stream)
{
    int st = check_conv_bwd(desc, x, xn, w, dy, dyn, cu_seqlens_dev, cu_seqlens_host, dx, dxn, dw);
    if (st != BDGDN_OK) return st;
    if (bdgdn_shortconv_bwd_workspace(desc) > kConvScratchBytes) return BDGDN_ERR_SCRATCH;
    float *part = nullptr;
    if (conv_noalloc_scratch(static_cast<hipStream_t>(stream), &part) != hipSuccess) return BDGDN_ERR_LAUNCH;
    return conv_bwd_launch(desc, x, xn, w, bias, dy, dyn, cu_seqlens_dev, dx, dxn, dw, dbias, part,
                           static_cast<hipStream_t>(stream));
}

}  // extern "C"
