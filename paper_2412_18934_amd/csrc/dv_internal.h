// Internal interface between the host engine (dv_engine.cpp) and the HIP
// kernels (dv_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#define DV_TREE_MAX 64
#define DV_GEMM_TILE 32     // logical output rows per workgroup tile
#define DV_ATTN_TILE 32     // keys per attention tile
#define DV_ATTN_WAVES 4     // waves per attention workgroup (MFMA path)
#define DV_ATTN_SPLIT_KEYS 256   // keys per workgroup of the fp32-cache attention

// Per-step description of the draft tree, uploaded once per step.
struct StepDesc {
    int32_t M;        // tree nodes
    int32_t P;        // committed length before the step
    int32_t Mpad;     // M rounded up to 16
    int32_t pad0;
    int32_t tokens[DV_TREE_MAX];
    int32_t parents[DV_TREE_MAX];
    int32_t pos[DV_TREE_MAX];
    int32_t depth[DV_TREE_MAX];
    uint64_t anc[DV_TREE_MAX];  // bit j set: node j is on node i's root path
};

// Result written by the acceptance kernel, copied back to the host.
struct DevAccept {
    int32_t accept_len;
    int32_t bonus;
    int32_t path[DV_TREE_MAX];
    int32_t argmax[DV_TREE_MAX];
};

enum GemmEpi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

// "Split layout" of an activation matrix [Mpad][K] (Mpad = 16 MT) for the
// MFMA projections: each fp32 value v is stored as bf16 hi = v truncated and
// lo = round-to-nearest-even(v - hi), in the B-operand order of
// v_mfma_f32_16x16x32_bf16: for k-step s (32 columns), token tile mt and
// part p (0 hi, 1 lo), a 1 KB block of 64 lanes x 8 values, lane
// 16 (k%32)/8 + m%16 holding columns 32 s + 8 ((k%32)/8) .. +8 of token m.
// Block (s, mt, p) starts at element ((s MT + mt) 2 + p) 512.
// Size: K/32 * MT * 2 * 512 bf16 = 64 K MT bytes.

// GEMM variants (MFMA path): waves per workgroup, k-steps per load batch
// and tiles per work unit; supported: {8, 4, 2}, {4, 8, 2}, {4, 8, 1}
// Workgroup shape of the MFMA projection kernel: nw waves, u k-steps per
// batch of loads, tp tiles sharing the activation operand.  Instantiated
// shapes: {8,4,2}, {4,8,2}, {4,4,4}, {4,8,1}.
struct GemmShape {
    int nw;
    int u;
    int tp;
};

struct GemmArgs {
    const void *w0, *w1, *w2;  // QKV: wq, wk, wv; SWIGLU: w_gate, w_up; else w0
    const uint16_t *packed;    // bf16 MFMA path: the matrices in tile order (see
                               // k_pack_tiles), read instead of w0..w2
    int32_t N;                 // rows of one matrix (d_model, d_ffn or vocab)
    int32_t K;                 // reduction length (row length of the matrices)
    int32_t n_tiles;           // tiles of DV_GEMM_TILE logical rows
    int32_t ks;                // split-K factor (RESID only; partials go to `part`)
    int32_t k_per_split;       // reduction elements per split (multiple of 32)
    int32_t n_units;           // n_tiles * ks work units, looped over by the grid
    const float *x;            // VALU path: activations [Mpad][K], rows >= M are zero
    const uint16_t *xs;        // MFMA path: the same activations pre-split (split layout)
    int32_t M, Mpad;
    float *out;                // QKV: q [Mpad][d]; RESID (ks == 1): x [.][N];
                               // SWIGLU: h [Mpad][N]; LOGITS: logits [M][N] or null
    uint16_t *out_split;       // SWIGLU: h in split layout instead of `out` when set
    void *kc, *vc;             // QKV: this layer's K/V cache [H][cap][hd]
    int32_t cap, P, hd;
    const float *rope_cos, *rope_sin;  // [max_ctx][hd/2]
    const int32_t *pos;        // QKV: device StepDesc.pos
    float *part;               // RESID, ks > 1: partial sums [ks][64][N], folded
                               // into the residual stream by the next k_rmsnorm
    const float *ssq;          // QKV, SWIGLU, LOGITS: sums of squares from k_rmsnorm;
    float eps;                 // outputs are scaled by 1/sqrt(sum/dn + eps) per token
    int32_t dn;
    float *arg_val;            // LOGITS: per-tile max    [64][n_tiles]
    int32_t *arg_idx;          // LOGITS: per-tile argmax [64][n_tiles]
};

// RMSNorm is split in two: k_rmsnorm completes the residual row (embedding
// gather or split-K fold), writes x * gain and the sum of squares of each of
// DV_NORM_SLICES column slices; the consuming projection multiplies its
// outputs by 1/sqrt(sum/d + eps), a per-token scalar that commutes with W.
#define DV_NORM_SLICES 16
#define DV_NORM_THREADS 128

struct NormArgs {
    float *x;                  // [Mpad][d] residual stream
    const void *embed;         // when set: x = embedding rows of the tokens first
    const float *part;         // when ks > 0: x += sum_s part[s][m][:] first
    int32_t ks;
    const void *gain;          // [d] weight dtype
    float *u;                  // [Mpad][d] x * gain (fp32), or
    uint16_t *us;              // the same in split layout when set
    float *ssq;                // [Mpad][DV_NORM_SLICES] sums of squares of x
    int32_t d;
    int32_t M;
    const int32_t *tokens;     // device: StepDesc.tokens
};

struct AttnArgs {
    const float *q;            // [Mpad][H*hd] rotated queries
    const void *kc, *vc;       // layer cache [H][cap][hd]
    int32_t cap, hd, H;
    int32_t keys_per_split, n_split;
    const StepDesc *sd;
    float *part_o;             // [H][n_split][64][hd]
    float *part_m, *part_l;    // [H][n_split][64]
    float *out;                // [Mpad][H*hd] fp32 output, or
    uint16_t *out_split;       // the output in split layout when set
};

struct AcceptArgs {
    const float *arg_val;      // [64][n_tiles]
    const int32_t *arg_idx;
    int32_t n_tiles;
    const StepDesc *sd;
    DevAccept *acc;
};

struct CommitArgs {
    void *kc, *vc;             // whole cache [L][H][cap][hd]
    int32_t LH, cap, hd, P, n;
    int32_t path[DV_TREE_MAX];
};

// launchers (dv_kernels.hip); each returns the launch status
// copy a projection's bf16 rows into MFMA tile order (init time)
hipError_t launch_pack(const GemmArgs &a, int epi, uint16_t *dst, hipStream_t s);
// workgroups of 256 threads one CU can hold for a GEMM variant (cached)
int gemm_blocks_per_cu(int epi, int weight_bf16, int use_mfma, int mt, GemmShape sh);
// ev_start/ev_stop (optional, both or neither): timestamps of this launch
hipError_t launch_gemm(const GemmArgs &a, int grid, int epi, int weight_bf16, int use_mfma,
                       GemmShape sh, hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop);
hipError_t launch_rmsnorm(const NormArgs &a, int Mpad, int weight_bf16, hipStream_t s);
hipError_t launch_attention(const AttnArgs &a, int kv_bf16, hipStream_t s);
hipError_t launch_attn_merge(const AttnArgs &a, int Mpad, hipStream_t s);
hipError_t launch_accept(const AcceptArgs &a, hipStream_t s);
hipError_t launch_kv_commit(const CommitArgs &a, int kv_bf16, hipStream_t s);
