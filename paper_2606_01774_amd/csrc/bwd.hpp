// bwd.hpp -- argument block and launcher of the two-stream training backward
// (bwd_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdgdn {

// Backward of the two-stream training forward (bwd_kernels.hip): from the seed states of
// the split schedule's clean scan, the noisy blocks (with the state-gradient-independent part
// of the clean blocks) in parallel, a reverse scan of the clean state gradient, the clean
// blocks in parallel.  Gradients are fp32; a workgroup runs the v-heads of a (block, q/k
// head) in turn, storing dq, dk for the first and adding for the others (deterministic).
struct BwdArgs {
    const void *q, *k, *v, *qn, *kn, *vn;   // bf16 [rows][heads][128]
    const float *g, *beta, *gn, *betan;      // [rows][h_v]
    const void *dout, *doutn;                // [rows][h_v][128] of the output type
    const _Float16 *seeds;                   // [global block][h_v][128][128] fp16
    const float *dht;                        // [seq][h_v][128][128] or null
    float *dq, *dk, *dv, *dg, *db;
    float *dqn, *dkn, *dvn, *dgn, *dbn;
    float *dh0;                              // or null
    _Float16 *cterm;                         // [global block][h_v][64 tiles][64 lanes][4]: the part of dh_(b-1)
                                             // that does not depend on dh_b (noisy seed gradient
                                             // + clean terms), fp16 like dh
    _Float16 *uk;                            // [global block][h_v][32][128]: U K of each clean block
    float *gnb;                              // [global block][h_v]: gamma_n of each clean block
    _Float16 *dh;                            // [global block][h_v][64 tiles][64 lanes][4]: gradient at
                                             // block ends (fp16, tile-native like cterm; may be cterm
                                             // itself: the scan reads cterm_b before writing dh_b)
    const float *range;                      // {sigma, 1 / sigma}: the upstream gradients enter the
                                             // fp16 operands times sigma, the fp32 results are
                                             // divided by it (launch_bwd_range writes them)
    const int32_t *cu;                       // packed documents, or null
    // one time segment of every chain (strided checkpoints): per sequence or document the
    // blocks blk0 .. blk0 + seg_len - 1, with workspace units numbered from seg[n] (clean
    // blocks) and noisy blocks of two sub-blocks from segp[n] (tables of sequences + 1
    // entries); carry [seq][h_v][128][128] fp32 hands the state gradient at the segment's
    // start to the segment before it; seg null: all blocks, units by global block
    const int *seg, *segp;
    float *carry;
    int blk0, seg_len;
    int n_docs;
    int n_chains;                            // sequences x v-heads
    long n_units;                            // global blocks x v-heads (set by launch_bwd)
    int T, nblk, L, h_qk, h_v;
    float scale;
};
// A further noisy view (the complementary-view backward): its inputs, the upstream gradient
// of its readout and its gradients, laid out as the noisy stream of BwdArgs.
struct BwdView {
    const void *q, *k, *v;
    const float *g, *beta;
    const void *dout;
    float *dq, *dk, *dv, *dg, *db;
};
// The range pass: max |x| over the upstream gradients (arr[0 .. count-1]: dO, dO~ of each view
// in the output type, then dht in fp32 when last_f32) into part[kRangeBlocks], reduced to
// range = {sigma, 1 / sigma}.
constexpr int kRangeArrays = 19, kRangeBlocks = 512;
struct RangeArgs {
    const void *arr[kRangeArrays];
    long n[kRangeArrays];   // elements of each array (multiples of 128)
    int count;
    bool last_f32;
    float *part;            // [kRangeBlocks]
    float *range;           // [2]
};
hipError_t launch_bwd_range(bool bf16_out, const RangeArgs &r, hipStream_t s);

// The per-step fp32 backward (bwd_generic.hip) for the shapes outside the block-form
// kernels: one call's arguments.
struct GenBwdCall {
    const void *q, *k, *v;
    const float *g, *beta;
    const void *dout;
    float *dq, *dk, *dv, *dg, *db;
    const void *qn, *kn, *vn;
    const float *gn, *betan;
    const void *doutn;
    float *dqn, *dkn, *dvn, *dgn, *dbn;
    const BwdView *more;
    int n_more;
    const int32_t *cu, *cu_host;   // packed documents (device, host), or null
    int n_seq;                     // sequences or documents
    long rows, total_blocks;       // token rows; blocks of all chains' sequences
    const float *h0, *dht;
    float *dh0;
    int T, L, h_qk, h_v, d_k, d_v;
    float scale;
    void *workspace;
};
size_t bwd_generic_workspace(int n_seq, long total_blocks, int h_v, int dk, int dv);
bool bwd_generic_supported(bool f32_in, int dk, int dv, int L, int n_views);
hipError_t launch_bwd_generic(bool f32_in, bool f32_out, const GenBwdCall &c, hipStream_t s);
size_t bwd_block_lds();
// The backward of a's two streams, plus n_more further noisy views seeded from the same clean
// states (their seed gradients summed into the clean state gradient).  a.L is the clean
// block; with n_pair_units > 0 every noisy block spans two clean blocks (n_pair_units =
// noisy blocks x v-heads).
hipError_t launch_bwd(bool bf16_out, const BwdArgs &a, const BwdView *more, int n_more, int n_chains,
                      long n_block_units, long n_pair_units, hipStream_t s);
// The segment tables of a segmented backward: for segments k = 0 .. n_seg - 1 of seg_len
// blocks of L positions, seg[k][n] = the blocks of sequences 0 .. n - 1 inside segment k and
// segp[k][n] = their noisy blocks of two sub-blocks (n = 0 .. n_seq); lengths from cu
// (packed) or T.
hipError_t launch_bwd_seg_plan(const int32_t *cu, int n_seq, int T, int L, int seg_len, int n_seg, int *seg,
                               int *segp, hipStream_t s);

}  // namespace bdgdn
