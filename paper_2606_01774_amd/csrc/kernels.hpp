// kernels.hpp -- argument blocks and host-side launchers of the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bdgdn {

constexpr int kMaxOrder = 512;  // documents whose longest-first order travels in the kernel arguments

struct FwdArgs {
    const void *q, *k, *v, *qn, *kn, *vn;
    const float *g, *beta, *gn, *betan;
    const int32_t *cu;   // device cu_seqlens or NULL
    const float *h0;
    float *ht;
    void *o, *on;
    int T, h_qk, h_v, dv, L;
    int n_chains, n_vt;  // chains = sequences x v-heads; d_v tiles per chain
    float scale;
    int n_order;         // 0, or the number of documents listed in order[]
    int order[kMaxOrder];
};

// Block-local UT transform (one workgroup per (block, v-head)).
struct IntraArgs {
    const void *q, *k, *qn, *kn;
    const float *g, *beta, *gn, *betan;
    unsigned char *ws;   // records, ((block * h_v) + h) * record bytes
    int T, L, nblk;      // tokens per sequence (packed: total), block, blocks per sequence
    long total_blocks;   // sequences * nblk
    int h_qk, h_v;
};

// Sequential scan (one workgroup per (chain, d_v tile)).
struct ScanArgs {
    const void *q, *k, *v, *qn, *kn, *vn;
    const float *g, *beta, *gn, *betan;   // read by the one-kernel schedule only
    const int32_t *cu;
    const float *h0;
    float *ht;
    void *o, *on;
    const unsigned char *ws;
    void *bs;            // seed states by (global block, v-head): fp32 (split schedule, views),
                         // fp16 (the backward's recomputation), or null
    int T, L, nblk, h_qk, h_v, dv;
    int nl;              // noisy block of the small-block one-kernel forward (L is its clean chunk)
    // one time segment of every chain (the backward's strided checkpoints; seeds kernels
    // only): blocks blk0 .. blk0 + seg_len - 1 of each sequence or document, whose seeds are
    // indexed from seg[sequence]; seg null: all blocks, indexed by global block
    const int *seg;
    int blk0, seg_len;
    int n_chains, n_vt;
    float scale;
    int n_order;
    int order[kMaxOrder];
};

// The chunk-parallel forward (chunked.hpp): a clean UT-record kernel and a state pass
// over the blocks before each chain's last segment, then one workgroup per (chain,
// segment) for the outputs.  Chains are (sequence or document, v-head); a chain of nb
// blocks has nseg = ceil(nb / G) segments of G blocks.
struct ChunkArgs {
    const void *q, *k, *v, *qn, *kn, *vn;
    const float *g, *beta, *gn, *betan;
    const int32_t *cu;      // packed documents (device), or null
    const float *h0;
    float *ht;
    void *o, *on;
    unsigned char *rec;     // clean UT records of the state pass
    float *ckpt;            // clean state at every segment start after the first
    int T, L, nblk, h_qk, h_v, dv;
    int G;                  // blocks per segment
    int n1;                 // chains' sequences / documents with two or more segments (the
                            // first n1 in processing order)
    int J_max;              // blocks of the longest state pass: (max nseg - 1) * G
    int n_groups;           // (position in order, segment, q/k head) groups of the out kernel
    int n_ot;               // d_v tiles of the out kernel
    int n_vt;               // 32-column tiles of the state pass
    float scale;
    int n_order;            // packed: documents listed in order[]
    int order[kMaxOrder];   // packed, longest first: doc | (segments of the documents before it) << 10
};

// Noisy-block pass of the split schedule (one workgroup per (global block, v-head)).
struct NoisyArgs {
    const void *qn, *kn, *vn;
    const float *gn, *betan;
    const float *bs;     // seed states [global block][h_v][d_k][d_v]
    const int32_t *cu;   // device cu_seqlens or NULL
    void *on;
    int T, L, nblk, n_docs;   // tokens per sequence (packed: total), block, blocks per sequence
    long total_blocks;
    int h_qk, h_v;
    float scale;
};

struct ServeArgs {
    const void *q, *k, *v;
    const float *g, *beta;
    float *pool;         // read (denoise) or read + written in place (commit)
    const int32_t *slot; // NULL: slot[r] = r
    void *o;             // NULL allowed for commit
    int R, h_qk, h_v, dv, L;
    int n_vt;
    float scale;
    float *states;       // recorded states [R][n_rec][h_v][d_k][d_v] (commit_record, accept), or NULL
    int n_rec;           // recorded positions: the block's last n_rec
    const int32_t *accept;   // accepted offsets [R] (accept)
};

// Element types of one call: inputs / MFMA operands / outputs.
enum class Types {
    BF16_IN_F32_OUT = 0,   // bf16 q,k,v staged as fp16 operands, fp32 outputs
    BF16_IN_BF16_OUT = 1,  // bf16 q,k,v staged as fp16 operands, bf16 outputs
    F32 = 2,               // fp32 end to end
};

// Each returns hipSuccess or the launch error.  lp is the padded block tile (16/32/64).
hipError_t launch_fwd_fused(Types ty, int dk, int lp, const FwdArgs &a, hipStream_t s);
hipError_t launch_denoise(Types ty, int dk, int lp, const ServeArgs &a, hipStream_t s);
hipError_t launch_commit(Types ty, int dk, int lp, bool with_o, const ServeArgs &a, hipStream_t s);
// The commit pass that also writes the states before the block's last n_rec positions
// (streaming kernels: bf16 inputs, d_k = d_v = 128, blocks of at most 32 positions).
bool record_supported(Types ty, int dk, int dv, int lp);
hipError_t launch_commit_record(Types ty, int lp, bool with_o, const ServeArgs &a, hipStream_t s);
// pool[slot[r]] <- states[r][accept[r]] for every head where accept[r] < n_rec.
hipError_t launch_accept_states(const ServeArgs &a, int dk, hipStream_t s);
// Two-kernel training forward (UT transform records, then the scan).
hipError_t launch_fwd_scan(Types ty, int dk, int lp, const IntraArgs &ia, const ScanArgs &sa, hipStream_t s);
// The one-kernel pipelined schedule (UT transform inside the scan workgroups): bf16
// inputs, blocks of at most 32 positions.
bool pipelined_supported(Types ty, int dk, int lp);
// clean_out = false: no clean outputs (a further noisy view of the complementary-view forward).
hipError_t launch_fwd_pipelined(Types ty, int dk, int lp, const ScanArgs &a, hipStream_t s, bool clean_out = true);
// Blocks of L = 2 a.L positions (L even, 34 .. 64) in the same kernel: the chain runs on
// sub-blocks of a.L positions and each noisy block spans two of them.
bool pair_supported(Types ty, int dk, int L);
hipError_t launch_fwd_pipelined_pair(Types ty, int dk, const ScanArgs &a, hipStream_t s, bool clean_out = true);
// Noisy blocks of a.nl = 1, 2, 4 or 8 positions in the same kernel: the chain runs on clean
// chunks of a.L = 32 positions, each holding 32 / a.nl noisy blocks.
bool small_supported(Types ty, int dk, int L);
hipError_t launch_fwd_pipelined_small(Types ty, int dk, const ScanArgs &a, hipStream_t s);
// The same, also writing the seed state of every (block, v-head) to a.bs (d_k = 128).
hipError_t launch_fwd_pipelined_seeds(Types ty, int lp, const ScanArgs &a, hipStream_t s);
// The split schedule (clean scan exposing the seed states, then the noisy-block pass):
// bf16 inputs, d_k = d_v = 128, blocks of at most 32 positions.
bool split_supported(Types ty, int dk, int dv, int lp);
hipError_t launch_fwd_split(Types ty, int lp, const ScanArgs &sa, const NoisyArgs &na, hipStream_t s);
size_t scan_record_bytes(Types ty, int lp);
int scan_tile_v();
// d_v columns handled by one workgroup of the training / serving kernels.
int fwd_tile_v();
int serve_tile_v();
// Whether the (types, d_k, lp) combination is instantiated and fits in LDS.
bool fwd_supported(Types ty, int dk, int lp);

// The split schedule's two kernels on their own: the clean scan writing every block's seed
// state (with f16_seeds: the backward's recomputation, fp16 seeds and no clean outputs), and
// the noisy-block pass from the seeds.
hipError_t launch_scan_states(int lp, bool f32_out, bool f16_seeds, const ScanArgs &sa, hipStream_t s);
hipError_t launch_noisy_blocks(int lp, bool f32_out, const NoisyArgs &na, hipStream_t s);

// The chunk-parallel forward: bf16 inputs, d_k = d_v in {64, 128}, blocks of at most 32.
bool chunked_supported(Types ty, int dk, int dv, int lp);
hipError_t launch_fwd_chunked(Types ty, int dk, int lp, const ChunkArgs &a, hipStream_t s);
// Columns of one workgroup of the out kernel: d_v (one tile) or 32.
bool chunk_tile_supported(int dk, int tile);
size_t chunk_rec_bytes(int lp);

// The two-stream ShortConv (conv_kernels.hip).  x, xn, y, yn, dy, dyn are [rows][D] of the
// conv dtype; w [D][W] and bias [D] fp32; part [row groups][W + 1][D] fp32 partials of the
// backward; n_rg is set by the launchers.
struct ConvArgs {
    const void *x, *xn, *dy, *dyn;
    const float *w, *bias;
    const int32_t *cu;   // [n_docs + 1] device offsets, or NULL for sequences of seqlen rows
    void *y, *yn;        // forward outputs, or dx, dxn in the backward
    float *part, *dw, *dbias;
    long rows;
    int D, L, act, n_docs, seqlen, n_rg;
};
size_t conv_part_floats(long rows, int D, int width);
// The no-allocation backward's fixed scratch: its size, and its device address on the
// device of `stream` (the current device for a NULL stream), looked up once per device.
constexpr size_t kConvScratchBytes = 32u << 20;
hipError_t conv_noalloc_scratch(hipStream_t stream, float **ptr);
hipError_t launch_shortconv_fwd(bool bf16, int width, const ConvArgs &a, hipStream_t s);
hipError_t launch_shortconv_bwd(bool bf16, int width, const ConvArgs &a, hipStream_t s);

}  // namespace bdgdn
