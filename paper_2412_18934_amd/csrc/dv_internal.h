// Internal interface between the host engine (dv_engine.cpp) and the HIP
// kernels (dv_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#define DV_TREE_MAX 64
#define DV_GEMM_TILE 32     // logical output rows per workgroup tile
#define DV_ATTN_TILE 32     // keys per attention tile

#define DV_ATTN_SPLIT_KEYS 256   // keys per workgroup of the fp32-cache attention

// Per-step description of the draft tree (host side; the kernels receive
// the parts they need by value in their arguments, so no kernel reads it
// from memory before it can address its inputs).
struct StepDesc {
    int32_t M;        // tree nodes
    int32_t P;        // committed length before the step
    int32_t Mpad;     // M rounded up to 16
    int32_t half;     // activations in the half split layout (M <= 8)
    int32_t tokens[DV_TREE_MAX];
    int32_t parents[DV_TREE_MAX];
    int32_t pos[DV_TREE_MAX];
    int32_t depth[DV_TREE_MAX];
    uint64_t anc[DV_TREE_MAX];  // bit j set: node j is on node i's root path
};

// The tree as attention needs it (by value).
struct TreeMask {
    int32_t M, P, Mpad, half;  // half: outputs in the half split layout
    uint64_t anc[DV_TREE_MAX];
};

// Result written by the acceptance kernel, copied back to the host.
struct DevAccept {
    int32_t accept_len;
    int32_t bonus;
    int32_t path[DV_TREE_MAX];
    int32_t argmax[DV_TREE_MAX];
};

// EPI_PLAIN: the sums themselves, out [M][N] fp32 (no input norm; the draft's
// gated fusion)
enum GemmEpi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3, EPI_PLAIN = 4 };

// "Split layout" of an activation matrix [Mpad][K] (Mpad = 16 MT) for the
// MFMA projections: each fp32 value v is stored as bf16 hi = v truncated and
// lo = round-to-nearest-even(v - hi), in the B-operand order of
// v_mfma_f32_16x16x32_bf16: for k-step s (32 columns), token tile mt and
// part p (0 hi, 1 lo), a 1 KB block of 64 lanes x 8 values, lane
// 16 (k%32)/8 + m%16 holding columns 32 s + 8 ((k%32)/8) .. +8 of token m.
// Block (s, mt, p) starts at element ((s MT + mt) 2 + p) 512.
// Size: K/32 * MT * 2 * 512 bf16 = 64 K MT bytes.
// Half layout (steps of at most 8 nodes, flag `half`, written as MT = 0):
// one 1 KB block per k-step, B-operand columns 0-7 holding the hi parts of
// tokens 0-7 and columns 8-15 their lo parts, so one MFMA covers both and
// the sums of columns n and n + 8 give token n.  Block s starts at element
// 512 s; a token's lo values sit 64 elements after its hi values.  Size:
// K/32 * 512 bf16 = 32 K bytes.

// Projection weights, MFMA path.  The output rows are cut into 16-row
// blocks; rb consecutive blocks form a row group (one work unit, or ks units
// when the reduction is split).  Weights are stored k-major: the 1 KB block
// of (k-step s, group g, block b) -- 16 rows x 32 columns in A-operand lane
// order, lane l holding row l%16, columns 32 s + 8 (l/16) .. +8 -- starts at
// element ((s G + g) rb + b) 512.  Blocks pair up into 32-row tiles (b even,
// b + 1) whose halves the epilogues combine:
//   QKV:    dims [j0, j0+16) of one head | dims j0+hd/2+[0,16) (rotary pairs),
//           segments q | k | v one after another;
//   SWIGLU: gate rows [16t, 16t+16) | the same up rows;
//   else:   rows [32t, 32t+16) | [32t+16, 32t+32).
// int8 weights use the same groups and blocks over pairs of k-steps: the 1 KB
// block of (k-step pair p, g, b) -- 16 rows x 64 columns, lane l holding row
// l%16, columns 64 p + 8 (l/16) .. +8 in bytes 0-7 and 64 p + 32 + 8 (l/16)
// .. +8 in bytes 8-15 -- starts at byte ((p G + g) rb + b) 1024; the row
// scales follow the packed row order (block gb = g rb + b, row r at gb 16 + r).
enum WeightKind { W_F32 = 0, W_BF16 = 1, W_I8 = 2 };

struct GemmArgs {
    const void *w0, *w1, *w2;  // QKV: wq, wk, wv; SWIGLU: w_gate, w_up; else w0
    const uint16_t *packed;    // MFMA path: the weights in block order (above)
    const float *s0, *s1, *s2; // int8: per-row scales of w0, w1, w2 (packing only)
    const float *scale;        // int8: the row scales in packed row order
    int32_t N;                 // rows of one matrix (d_model, d_ffn or vocab)
    int32_t K;                 // reduction length (row length of the matrices)
    int32_t n_tiles;           // 32-row tiles (QKV counts the three matrices)
    int32_t rb;                // MFMA path: 16-row blocks per row group (2 or 4)
    int32_t n_groups;          // row groups: MFMA 2 n_tiles / rb; VALU n_tiles
    int32_t ks;                // K splits per row group (RESID, MFMA path only)
    int32_t n_units;           // n_groups * ks
    const float *x;            // VALU path: activations [Mpad][K], fp32
    const uint16_t *xs;        // MFMA path: the same activations in split layout
    int32_t M, Mpad;
    int32_t half;              // xs, us and out_split in the half split layout
    float *out;                // QKV: q [Mpad][d]; SWIGLU: h [Mpad][N] (VALU
                               // consumer); LOGITS: logits [M][N] or null
    uint16_t *out_split;       // SWIGLU: h in split layout (MFMA consumer)
    void *kc, *vc;             // QKV: this layer's K/V cache
    int32_t cap, P, hd;
    const float *rope_cos, *rope_sin;  // [max_ctx][hd/2]
    int32_t pos[DV_TREE_MAX];  // QKV: position P + depth - 1 of each node
    // input normalisation (QKV, SWIGLU, LOGITS): the activations are x * gain
    // of an RMSNorm whose 1/rms, a per-token scalar that commutes with W, is
    // applied to the outputs: 1/sqrt(sum_j ssq_in[m][j] / dn + eps)
    const float *ssq_in;       // [Mpad][n_ssq_in] partial sums of squares
    int32_t n_ssq_in;
    float eps;
    int32_t dn;
    // RESID: the residual stream x [Mpad][N] += W a; then the next RMSNorm's
    // numerator x * gain is written for the consuming projection, with the
    // per-group sums of squares of x
    float *resid;
    const void *gain;          // [N], weight dtype
    float *u;                  // x * gain, fp32 [Mpad][N] (VALU consumer), or
    uint16_t *us;              // in split layout (MFMA consumer)
    float *ssq_out;            // [Mpad][n_groups]
    float *part;               // ks > 1: per-unit partial sums
    uint32_t *cnt;             // ks > 1: arrivals per row group, 0 between launches
    float *arg_val;            // LOGITS: per-group max    [64][n_groups]
    int32_t *arg_idx;          // LOGITS: per-group argmax [64][n_groups]
};

// Workgroup shape of the MFMA projection kernel: nw waves, u k-steps of loads
// in flight per wave.  Instantiated: {4, 2} with rb 4, {4, 4} with rb 2.
struct GemmShape {
    int nw;
    int u;
};

// The first RMSNorm of a step (on the token embeddings): k_embed_norm
// gathers the rows into the residual stream, writes x * gain for the first
// projection and the sums of squares of DV_NORM_SLICES column slices.
#define DV_NORM_SLICES 16
#define DV_NORM_THREADS 128

struct NormArgs {
    float *x;                  // [Mpad][d] residual stream (written)
    const float *x_in;         // [M][d] input rows instead of embeddings, or null
    const void *embed;         // [V][d] token embeddings, weight dtype
    const void *gain;          // [d] weight dtype
    float *u;                  // [Mpad][d] x * gain (fp32), or
    uint16_t *us;              // the same in split layout when set
    float *ssq;                // [Mpad][DV_NORM_SLICES] sums of squares of x
    int32_t d;
    int32_t M;
    int32_t half;              // us in the half split layout
    int32_t tokens[DV_TREE_MAX];  // token ids of the nodes
};

struct AttnArgs {
    const float *q;            // [Mpad][H*hd] rotated queries
    const void *kc, *vc;       // layer cache [H][cap][hd]
    int32_t cap, hd, H;
    int32_t keys_per_split, n_split;
    TreeMask tm;
    float *part_o;             // [H][n_split][64][hd] unnormalised split outputs
    float *part_m, *part_l;    // [H][n_split][64] their running max (base 2) and sum
    uint32_t *cnt;             // [H] arrivals of the splits, 0 between launches
    float *out;                // [Mpad][H*hd] fp32 output, or
    uint16_t *out_split;       // the output in split layout when set
};

struct AcceptArgs {
    const float *arg_val;      // [64][n_parts] per-group (max, argmax) of the logits
    const int32_t *arg_idx;
    int32_t n_parts;
    int32_t M, Mpad;
    int32_t tokens[DV_TREE_MAX], parents[DV_TREE_MAX], depth[DV_TREE_MAX];
    DevAccept *acc;
};

// Sampled acceptance (one workgroup): the tree walk of the speculative
// sampling rule over full-vocabulary rows of logits and draft probabilities.
struct SampleArgs {
    const float *logits;       // [M][V]
    const float *q;            // [M][V] draft distributions
    float *p;                  // [V] workspace: the current (residual) distribution
    int32_t V, M;
    float inv_t;               // 1 / temperature
    int32_t tokens[DV_TREE_MAX], parents[DV_TREE_MAX];
    float u_accept[DV_TREE_MAX], u_bonus[DV_TREE_MAX];
    DevAccept *acc;
};

struct CommitArgs {
    void *kc, *vc;             // whole cache [L][H][cap][hd]
    int32_t LH, cap, hd, P, n;
    int32_t path[DV_TREE_MAX];
};

// launchers (dv_kernels.hip); each returns the launch status
// copy a projection's bf16 rows into MFMA block order (init time)
hipError_t launch_pack(const GemmArgs &a, int epi, int wkind, void *dst, hipStream_t s);
hipError_t launch_pack_scales(const GemmArgs &a, int epi, float *dst, hipStream_t s);
// the MFMA workgroup shape used for row groups of rb blocks
GemmShape gemm_shape(int rb);
// workgroups one CU can hold for a GEMM variant (cached)
int gemm_blocks_per_cu(int epi, int wkind, int use_mfma, int mt, int rb);
// whether an MFMA projection variant with 8-block row groups exists for this
// epilogue, weight kind and token-tile count
bool gemm_has_rb8(int epi, int wkind, int mt);
// ev_start/ev_stop (optional, both or neither): timestamps of this launch
hipError_t launch_gemm(const GemmArgs &a, int grid, int epi, int wkind, int use_mfma,
                       hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop);
hipError_t launch_embed_norm(const NormArgs &a, int Mpad, int weight_bf16, hipStream_t s);
hipError_t launch_attention(const AttnArgs &a, int kv_bf16, hipStream_t s);
hipError_t launch_attn_merge(const AttnArgs &a, int Mpad, hipStream_t s);
hipError_t launch_accept(const AcceptArgs &a, hipStream_t s);
hipError_t launch_accept_sampled(const SampleArgs &a, hipStream_t s);

// Allocation-free sampled acceptance: the kernel's workspace is a fixed device
// array of the library (one copy per GPU): the result struct in its first
// DV_NOALLOC_ACC_BYTES, then the two distribution rows of up to
// DV_NOALLOC_MAX_VOCAB floats each.
#define DV_NOALLOC_ACC_BYTES 1024
#define DV_NOALLOC_SCRATCH_BYTES (DV_NOALLOC_ACC_BYTES + 2 * 4 * (size_t)DV_NOALLOC_MAX_VOCAB)
#define DV_NOALLOC_MAX_DEVICES 64
// device address of that array on the current device (looked up once per
// device with hipGetSymbolAddress)
hipError_t noalloc_scratch(void **out);

// Large-M prefill (bf16 weights, MFMA path): the chunk's activations in split
// layout of MT = Mp / 16 token tiles (Mp a multiple of 128), norms applied
// by their consumers from sums of squares over 64-row slices ([Mp][d / 64]).
struct PfArgs {
    const uint16_t *packed;  // weights in block order
    int NB;                  // 16-row blocks of the matrix
    int K;                   // reduction length (multiple of 32)
    const uint16_t *xs;      // activations, split layout of MT token tiles
    int MT;                  // token tiles of the split layout (Mp / 16)
    int M;                   // real tokens (the rest is padding)
    int P0;                  // cache slot / position of token 0
    // input norm (QKV, SWIGLU): rinv = 1/sqrt(sum_j ssq_in[m][j] / d + eps)
    const float *ssq_in;
    int nsq_in;
    float eps;
    int d;                   // d_model
    // QKV
    float *q;                // [Mp][d] rotated queries
    void *kc, *vc;           // this layer's cache
    int cap, hd;
    const float *rope_cos, *rope_sin;
    // SWIGLU: h in split layout (K = F)
    uint16_t *hs;
    // RESID: x [Mp][d] += sums; us = x * gain (split layout), ssq_out [Mp][d / 64]
    float *x;
    const uint16_t *gain;
    uint16_t *us;
    float *ssq_out;
};

// embedding rows, the first norm's numerator (split layout) and its sums of squares
hipError_t launch_pf_embed(const int32_t *tokens, const void *embed, int M, int Mp, int d, const void *gain, float *x,
                           uint16_t *us, float *ssq, hipStream_t s);
// the prefill GEMM with the EPI_QKV, EPI_SWIGLU or EPI_RESID epilogue
hipError_t launch_pf_gemm(const PfArgs &a, int epi, hipStream_t s);
// causal attention of the chunk; output in split layout (MT token tiles)
hipError_t launch_attn_causal(const float *q, const void *kc, const void *vc, int M, int P0, int H, int hd, int cap,
                              int MT, uint16_t *out, hipStream_t s);

// Draft side
#define DV_TOPK_MAX 16
struct DgfTokens {
    int32_t tok[DV_TREE_MAX];
};
struct RowIndex {
    int32_t idx[DV_TREE_MAX];
};
struct TopkArgs {
    int32_t rows[DV_TREE_MAX];  // logits rows to rank
    int32_t k;
    int32_t *out_tok;           // [rows][DV_TOPK_MAX]
    float *out_p;               // [rows][DV_TOPK_MAX]
};
// DGF: the n feature rows and token embeddings as split-layout operands of
// K = d (rows n..Mpad zero); the gate input [h1 || h2] (K = 2 d); the mix
// x0 = g h1 + (1 - g) h2 with g = sigmoid(z)
hipError_t launch_dgf_in(const float *feat, const void *embed, const DgfTokens &t, int n, int Mpad, int d,
                         uint16_t *xf, uint16_t *xe, hipStream_t s);
hipError_t launch_dgf_gate_in(const float *h1, const float *h2, int n, int Mpad, int d, uint16_t *xg, hipStream_t s);
hipError_t launch_dgf_mix(const float *z, const float *h1, const float *h2, int n, int d, float *x0, hipStream_t s);
hipError_t launch_gather_rows(const float *src, const RowIndex &ix, int n, int d, float *dst, hipStream_t s);
hipError_t launch_topk_probs(const float *logits, int V, const TopkArgs &a, int n_rows, hipStream_t s);

hipError_t launch_kv_commit(const CommitArgs &a, int kv_bf16, hipStream_t s);
