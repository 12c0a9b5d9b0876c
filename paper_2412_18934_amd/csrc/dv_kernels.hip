// HIP kernels (gfx950 / CDNA4) for one tree-verification step.
//
// Step structure (Section 3.1 of the paper: one forward pass of the target
// over the candidate tokens, then the acceptance rule):
//   k_rmsnorm        embedding gather (first layer) + RMSNorm -> fp32 rows
//   k_gemm_*         weight-streaming projections with fused epilogues:
//                      QKV    -> rotary embedding, q store, K/V cache write
//                      RESID  -> residual add into the fp32 stream (O, down)
//                      SWIGLU -> silu(gate) * up
//                      LOGITS -> logits + per-tile argmax
//   k_attn / merge   tree-masked attention over the cache, split over keys
//   k_accept         vocab-wide argmax reduce + greedy acceptance walk
//   k_kv_commit      in-place compaction of the accepted path
//
// Weights are bf16 or fp32, activations and accumulation fp32.  Every
// reduction runs in a fixed order, so results are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "dv_internal.h"

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// scalar helpers

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16 bits, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f2bf(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ float load(const float *p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float *p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t *p, size_t i) { return bf2f(p[i]); }
    static __device__ __forceinline__ void store(uint16_t *p, size_t i, float v) { p[i] = f2bf(v); }
};

// ---------------------------------------------------------------------------
// GEMM tile -> weight rows
//
// A workgroup tile has DV_GEMM_TILE = 32 logical rows made of two halves of
// 16.  The halves map to physical rows so that each epilogue finds the pair
// of values it needs in the same tile:
//   QKV:    half 0 = dims [j0, j0+16) of one head, half 1 = dims j0+hd/2+..
//           (the rotary pairs), segments q | k | v one after another;
//   SWIGLU: half 0 = gate rows [16t, 16t+16), half 1 = the same up rows;
//   else:   rows [32t, 32t+32) of w0.

struct RowMap {
    const void *ptr[2];
    int32_t row0[2];
};

__device__ __forceinline__ RowMap row_map(const GemmArgs &a, int epi, int t)
{
    RowMap m;
    if (epi == EPI_QKV) {
        const int per_seg = a.N / DV_GEMM_TILE;
        const int seg = t / per_seg, tt = t - seg * per_seg;
        const int per_head = a.hd / DV_GEMM_TILE;
        const int h = tt / per_head, j0 = (tt - h * per_head) * 16;
        const void *w = seg == 0 ? a.w0 : (seg == 1 ? a.w1 : a.w2);
        m.ptr[0] = m.ptr[1] = w;
        m.row0[0] = h * a.hd + j0;
        m.row0[1] = h * a.hd + a.hd / 2 + j0;
    } else if (epi == EPI_SWIGLU) {
        m.ptr[0] = a.w0;
        m.ptr[1] = a.w1;
        m.row0[0] = m.row0[1] = t * 16;
    } else {
        m.ptr[0] = m.ptr[1] = a.w0;
        m.row0[0] = t * DV_GEMM_TILE;
        m.row0[1] = t * DV_GEMM_TILE + 16;
    }
    return m;
}

// ---------------------------------------------------------------------------
// GEMM epilogues on the tile in LDS
//
// tileY[m][r] (m < Mpad, r < 32) holds one work unit's sums.  A tile is
// owned by exactly one workgroup unless the projection is split over K
// (RESID only): then each split stores its partial tile and the next
// k_rmsnorm adds the splits into the residual stream in split order, so no
// workgroup ever waits for another and the sum order is fixed.

#define TILE_LD (DV_GEMM_TILE + 1)

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

template <int EPI, typename KV>
__device__ void gemm_epilogue(const GemmArgs &a, float (*tileY)[TILE_LD], int t, int ksl)
{
    const int tid = threadIdx.x;
    if (EPI == EPI_RESID) {
        if (a.ks > 1) {
            float *dst = a.part + (size_t)ksl * DV_TREE_MAX * a.N + t * DV_GEMM_TILE;
            for (int e = tid; e < a.M * DV_GEMM_TILE; e += blockDim.x) {
                const int m = e / DV_GEMM_TILE, r = e % DV_GEMM_TILE;
                dst[(size_t)m * a.N + r] = tileY[m][r];
            }
        } else {
            for (int e = tid; e < a.M * DV_GEMM_TILE; e += blockDim.x) {
                const int m = e / DV_GEMM_TILE, r = e % DV_GEMM_TILE;
                a.out[(size_t)m * a.N + t * DV_GEMM_TILE + r] += tileY[m][r];
            }
        }
    } else if (EPI == EPI_SWIGLU) {
        for (int e = tid; e < a.Mpad * 16; e += blockDim.x) {
            const int m = e / 16, r = e % 16;
            a.out[(size_t)m * a.N + t * 16 + r] = silu(tileY[m][r]) * tileY[m][16 + r];
        }
    } else if (EPI == EPI_QKV) {
        const int per_seg = a.N / DV_GEMM_TILE;
        const int seg = t / per_seg, tt = t - seg * per_seg;
        const int per_head = a.hd / DV_GEMM_TILE;
        const int h = tt / per_head, j0 = (tt - h * per_head) * 16;
        const int half = a.hd / 2;
        for (int e = tid; e < a.M * 16; e += blockDim.x) {
            const int m = e / 16, r = e % 16;
            const int j = j0 + r;
            float y1 = tileY[m][r], y2 = tileY[m][16 + r];
            if (seg < 2) {
                const int pos = a.pos[m];  // P + depth(m) - 1
                const float c = a.rope_cos[(size_t)pos * half + j];
                const float s = a.rope_sin[(size_t)pos * half + j];
                const float o1 = y1 * c - y2 * s, o2 = y2 * c + y1 * s;
                y1 = o1;
                y2 = o2;
            }
            if (seg == 0) {
                a.out[(size_t)m * a.N + h * a.hd + j] = y1;
                a.out[(size_t)m * a.N + h * a.hd + j + half] = y2;
            } else {
                KV *c = reinterpret_cast<KV *>(seg == 1 ? a.kc : a.vc);
                const size_t row = ((size_t)h * a.cap + a.P + m) * a.hd;
                Elem<KV>::store(c, row + j, y1);
                Elem<KV>::store(c, row + j + half, y2);
            }
        }
    } else {  // EPI_LOGITS
        if (a.out) {
            for (int e = tid; e < a.M * DV_GEMM_TILE; e += blockDim.x) {
                const int m = e / DV_GEMM_TILE, r = e % DV_GEMM_TILE;
                a.out[(size_t)m * a.N + t * DV_GEMM_TILE + r] = tileY[m][r];
            }
        }
        if (tid < a.M) {
            float best = tileY[tid][0];
            int bi = 0;
            for (int r = 1; r < DV_GEMM_TILE; ++r) {
                const float v = tileY[tid][r];
                if (v > best) { best = v; bi = r; }
            }
            a.arg_val[(size_t)tid * a.n_tiles + t] = best;
            a.arg_idx[(size_t)tid * a.n_tiles + t] = t * DV_GEMM_TILE + bi;
        }
    }
}

// ---------------------------------------------------------------------------
// MFMA GEMM for bf16 weights.
//
// v_mfma_f32_16x16x32_bf16: A = 16 weight rows x 32 k, B = 32 k x 16 tokens.
// Lane l supplies A[l%16][8(l/16)..+8] (16 contiguous bytes of one weight
// row) and B[8(l/16)..+8][l%16] (8 fp32 activations of token l%16, split
// into bf16 hi + lo so the product keeps ~16 mantissa bits; two MFMAs per
// operand pair).  D: lane l holds rows 4(l/16)..+4 of token l%16.
//
// Work unit = (tile, K split).  The grid is sized to stay resident and
// loops over units; within a unit the four waves take contiguous quarters
// of the K range, U k-steps per batch of loads, and their accumulators are
// summed in LDS in wave order.

template <int MT> struct MfmaCfg { static constexpr int U = MT == 1 ? 8 : (MT == 2 ? 4 : 2); };

__device__ __forceinline__ void split_hi_lo(const float4 &a, const float4 &b, bf16x8 &hi, bf16x8 &lo)
{
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float h = __uint_as_float(__float_as_uint(v[i]) & 0xffff0000u);
        hi[i] = (__bf16)h;
        lo[i] = (__bf16)(v[i] - h);
    }
}

// Weight tiles in MFMA order.  For tile t, k-step s (32 columns) and half h,
// the 16 x 32 block is stored as 1 KB in lane order: lane l's 16 bytes are
// row row0[h] + l%16, columns 32 s + 8 (l/16) .. +8.  Blocks are ordered
// (t, s, h), so one wave's load instruction reads 1 KB contiguous and a
// wave walking its k range streams one contiguous region.

__global__ __launch_bounds__(128) void k_pack_tiles(GemmArgs a, int epi, uint16_t *dst)
{
    const int t = blockIdx.x, h = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int S = a.K / 32;
    const RowMap rm = row_map(a, epi, t);
    const uint16_t *src = reinterpret_cast<const uint16_t *>(rm.ptr[h]) +
                          (size_t)(rm.row0[h] + (lane & 15)) * a.K + (lane >> 4) * 8;
    for (int s = blockIdx.y; s < S; s += gridDim.y) {
        const uint4 v = *reinterpret_cast<const uint4 *>(src + 32 * s);
        *reinterpret_cast<uint4 *>(dst + (((size_t)t * S + s) * 2 + h) * 512 + lane * 8) = v;
    }
}

template <int MT, int N_STEPS>
__device__ __forceinline__ void mfma_steps(const uint16_t *wtile, const float *const *xrow,
                                           int k, f32x4 (&acc)[2][MT])
{
    u32x4 wa[N_STEPS][2];
    float4 xa[N_STEPS][MT][2];
#pragma unroll
    for (int u = 0; u < N_STEPS; ++u) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
            wa[u][h] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(wtile + (2 * u + h) * 512));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            xa[u][mt][0] = *reinterpret_cast<const float4 *>(xrow[mt] + k + 32 * u);
            xa[u][mt][1] = *reinterpret_cast<const float4 *>(xrow[mt] + k + 32 * u + 4);
        }
    }
#pragma unroll
    for (int u = 0; u < N_STEPS; ++u) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            bf16x8 hi, lo;
            split_hi_lo(xa[u][mt][0], xa[u][mt][1], hi, lo);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const bf16x8 w = __builtin_bit_cast(bf16x8, wa[u][h]);
                acc[h][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, hi, acc[h][mt], 0, 0, 0);
                acc[h][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, lo, acc[h][mt], 0, 0, 0);
            }
        }
    }
}

template <int MT, int EPI, typename KV>
__global__ __launch_bounds__(256) void k_gemm_mfma(GemmArgs a)
{
    constexpr int U = MfmaCfg<MT>::U;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rl = lane & 15, g = lane >> 4;
    const int K = a.K, S = K / 32;
    __shared__ float red[4][2][MT][4][64];
    __shared__ float tileY[DV_TREE_MAX][TILE_LD];

    for (int unit = blockIdx.x; unit < a.n_units; unit += gridDim.x) {
        const int t = unit / a.ks, ksl = unit - t * a.ks;
        const float *xrow[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xrow[mt] = a.x + (size_t)(mt * 16 + rl) * K + g * 8;
        const int kb = ksl * a.k_per_split;
        const int nsteps = (min(K, kb + a.k_per_split) - kb) / 32;
        const int s0 = (wave * nsteps) >> 2, s1 = ((wave + 1) * nsteps) >> 2;
        const uint16_t *wt = a.packed + ((size_t)t * S + kb / 32) * 1024 + lane * 8;

        f32x4 acc[2][MT];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[h][mt] = (f32x4){0.f, 0.f, 0.f, 0.f};
        int s = s0;
        for (; s + U <= s1; s += U) mfma_steps<MT, U>(wt + (size_t)s * 1024, xrow, kb + 32 * s, acc);
        for (; s < s1; ++s) mfma_steps<MT, 1>(wt + (size_t)s * 1024, xrow, kb + 32 * s, acc);

#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int j = 0; j < 4; ++j) red[wave][h][mt][j][lane] = acc[h][mt][j];
        __syncthreads();
        for (int e = threadIdx.x; e < 2 * MT * 4 * 64; e += 256) {
            const int l = e & 63, j = (e >> 6) & 3, mt = (e >> 8) % MT, h = (e >> 8) / MT;
            const float v = ((red[0][h][mt][j][l] + red[1][h][mt][j][l]) + red[2][h][mt][j][l]) +
                            red[3][h][mt][j][l];
            tileY[mt * 16 + (l & 15)][h * 16 + 4 * (l >> 4) + j] = v;
        }
        __syncthreads();
        gemm_epilogue<EPI, KV>(a, tileY, t, ksl);
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// VALU GEMM (fp32 weights, or bf16 where K is not a multiple of 32).
// Thread (row r = tid/8, lane-in-row kl = tid%8) walks k = kb + 8 kl + 64 i,
// 8 weights per load; 16 tokens per pass; the 8 partial sums of a row are
// combined with butterfly shuffles.

template <typename W> struct Load8;
template <> struct Load8<float> {
    static __device__ __forceinline__ void get(const float *p, float *o)
    {
        const float4 a = *reinterpret_cast<const float4 *>(p);
        const float4 b = *reinterpret_cast<const float4 *>(p + 4);
        o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
        o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
    }
};
template <> struct Load8<uint16_t> {
    static __device__ __forceinline__ void get(const uint16_t *p, float *o)
    {
        const uint4 v = *reinterpret_cast<const uint4 *>(p);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[2 * i] = __uint_as_float(w[i] << 16);
            o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
};

template <typename W, int EPI, typename KV>
__global__ __launch_bounds__(256) void k_gemm_valu(GemmArgs a)
{
    const int r = threadIdx.x >> 3, kl = threadIdx.x & 7;
    const int K = a.K;
    __shared__ float tileY[DV_TREE_MAX][TILE_LD];
    for (int unit = blockIdx.x; unit < a.n_units; unit += gridDim.x) {
        const int t = unit / a.ks, ksl = unit - t * a.ks;
        const RowMap rm = row_map(a, EPI, t);
        const int hsel = r >> 4;
        const W *wrow = reinterpret_cast<const W *>(rm.ptr[hsel]) + (size_t)(rm.row0[hsel] + (r & 15)) * K;
        const int kb = ksl * a.k_per_split;
        const int ke = min(K, kb + a.k_per_split);
        for (int m0 = 0; m0 < a.Mpad; m0 += 16) {
            float acc[16];
#pragma unroll
            for (int m = 0; m < 16; ++m) acc[m] = 0.f;
            for (int k = kb + kl * 8; k < ke; k += 64) {
                float w[8];
                Load8<W>::get(wrow + k, w);
#pragma unroll
                for (int m = 0; m < 16; ++m) {
                    float xv[8];
                    Load8<float>::get(a.x + (size_t)(m0 + m) * K + k, xv);
                    float s = acc[m];
#pragma unroll
                    for (int i = 0; i < 8; ++i) s = fmaf(w[i], xv[i], s);
                    acc[m] = s;
                }
            }
#pragma unroll
            for (int m = 0; m < 16; ++m) {
                float v = acc[m];
                v += __shfl_xor(v, 1);
                v += __shfl_xor(v, 2);
                v += __shfl_xor(v, 4);
                if (kl == 0) tileY[m0 + m][r] = v;
            }
        }
        __syncthreads();
        gemm_epilogue<EPI, KV>(a, tileY, t, ksl);
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// RMSNorm, one workgroup per token row (rows in [M, Mpad) are written as 0).
// Before normalising, the row of the residual stream is completed: either
// gathered from the embedding table (first layer) or incremented by the
// split-K partial sums of the projection that produced it, in split order.
// 256 threads x 4 consecutive floats per pass.

template <typename W>
__global__ __launch_bounds__(256) void k_rmsnorm(NormArgs a)
{
    const int m = blockIdx.x, tid = threadIdx.x, d = a.d;
    float *urow = a.u + (size_t)m * d;
    float *xrow = a.x + (size_t)m * d;
    if (m >= a.M) {
        for (int i = 4 * tid; i < d; i += 1024) {
            *reinterpret_cast<float4 *>(urow + i) = make_float4(0.f, 0.f, 0.f, 0.f);
            if (a.embed) *reinterpret_cast<float4 *>(xrow + i) = make_float4(0.f, 0.f, 0.f, 0.f);
        }
        return;
    }
    constexpr int MAXV = 8;  // d <= 8 * 1024
    float4 v[MAXV];
    const W *e = a.embed ? reinterpret_cast<const W *>(a.embed) + (size_t)a.tokens[m] * d : nullptr;
#pragma unroll
    for (int c = 0; c < MAXV; ++c) {
        const int i = 4 * tid + 1024 * c;
        if (i < d) {
            if (e) {
                v[c] = make_float4(Elem<W>::load(e, i), Elem<W>::load(e, i + 1),
                                   Elem<W>::load(e, i + 2), Elem<W>::load(e, i + 3));
            } else {
                v[c] = *reinterpret_cast<const float4 *>(xrow + i);
            }
        }
    }
    for (int s = 0; s < a.ks; ++s) {
        const float *p = a.part + ((size_t)s * DV_TREE_MAX + m) * d;
#pragma unroll
        for (int c = 0; c < MAXV; ++c) {
            const int i = 4 * tid + 1024 * c;
            if (i < d) {
                const float4 q = *reinterpret_cast<const float4 *>(p + i);
                v[c].x += q.x; v[c].y += q.y; v[c].z += q.z; v[c].w += q.w;
            }
        }
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < MAXV; ++c) {
        const int i = 4 * tid + 1024 * c;
        if (i < d) {
            if (e || a.ks) *reinterpret_cast<float4 *>(xrow + i) = v[c];
            ss = fmaf(v[c].x, v[c].x, ss);
            ss = fmaf(v[c].y, v[c].y, ss);
            ss = fmaf(v[c].z, v[c].z, ss);
            ss = fmaf(v[c].w, v[c].w, ss);
        }
    }
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    __shared__ float wsum[4];
    if ((tid & 63) == 0) wsum[tid >> 6] = ss;
    __syncthreads();
    const float tot = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
    const float rinv = 1.0f / sqrtf(tot / (float)d + a.eps);
    const W *gp = reinterpret_cast<const W *>(a.gain);
#pragma unroll
    for (int c = 0; c < MAXV; ++c) {
        const int i = 4 * tid + 1024 * c;
        if (i < d) {
            float4 o;
            o.x = v[c].x * rinv * Elem<W>::load(gp, i);
            o.y = v[c].y * rinv * Elem<W>::load(gp, i + 1);
            o.z = v[c].z * rinv * Elem<W>::load(gp, i + 2);
            o.w = v[c].w * rinv * Elem<W>::load(gp, i + 3);
            *reinterpret_cast<float4 *>(urow + i) = o;
        }
    }
}

// ---------------------------------------------------------------------------
// Tree-masked attention, split over keys (flash-decoding style).
// Workgroup (split s, head h) covers keys [s*kps, (s+1)*kps) of the P + M
// cache slots; the tree's own keys were written to slots P.. by the QKV
// epilogue.  Key j is visible to node i iff j < P or bit (j-P) of anc(i).
// Queries are handled 16 at a time; K/V tiles of 32 keys sit in LDS as fp32;
// an online softmax keeps (max, sum, o) per query.  Outputs per split:
// o (unnormalised), running max and sum.

template <int HD, typename KV>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a)
{
    constexpr int DPT = HD / 16;  // output dims per thread
    const int split = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const StepDesc *sd = a.sd;
    const int M = sd->M, P = sd->P, total = P + M;
    const int kb = split * a.keys_per_split;
    const int ke = min(total, kb + a.keys_per_split);
    const float scale = 1.0f / sqrtf((float)HD);
    const KV *kc = reinterpret_cast<const KV *>(a.kc) + (size_t)h * a.cap * HD;
    const KV *vc = reinterpret_cast<const KV *>(a.vc) + (size_t)h * a.cap * HD;
    const int D = a.H * HD;

    __shared__ float qs[16][HD];
    __shared__ float kt[DV_ATTN_TILE][HD + 1];
    __shared__ float vt[DV_ATTN_TILE][HD];
    __shared__ float sc[16][DV_ATTN_TILE + 1];
    __shared__ float mrun[16], lrun[16], alph[16];

    const int qi = tid >> 4, dd = (tid & 15) * DPT;
    for (int q0 = 0; q0 < M; q0 += 16) {
        const int nq = min(16, M - q0);
        for (int e = tid; e < 16 * HD; e += 256) {
            const int i = e / HD, d = e % HD;
            qs[i][d] = i < nq ? a.q[(size_t)(q0 + i) * D + h * HD + d] : 0.f;
        }
        if (tid < 16) { mrun[tid] = -INFINITY; lrun[tid] = 0.f; }
        float o[DPT];
#pragma unroll
        for (int c = 0; c < DPT; ++c) o[c] = 0.f;
        __syncthreads();

        for (int t0 = kb; t0 < ke; t0 += DV_ATTN_TILE) {
            const int nk = min(DV_ATTN_TILE, ke - t0);
            for (int e = tid; e < DV_ATTN_TILE * HD; e += 256) {
                const int j = e / HD, d = e % HD;
                float kv = 0.f, vv = 0.f;
                if (j < nk) {
                    kv = Elem<KV>::load(kc, (size_t)(t0 + j) * HD + d);
                    vv = Elem<KV>::load(vc, (size_t)(t0 + j) * HD + d);
                }
                kt[j][d] = kv;
                vt[j][d] = vv;
            }
            __syncthreads();
            for (int e = tid; e < 16 * DV_ATTN_TILE; e += 256) {
                const int i = e / DV_ATTN_TILE, j = e % DV_ATTN_TILE;
                const int key = t0 + j;
                bool vis = i < nq && j < nk;
                if (vis && key >= P) vis = (sd->anc[q0 + i] >> (key - P)) & 1ull;
                float s = -INFINITY;
                if (vis) {
                    float acc = 0.f;
#pragma unroll 8
                    for (int d = 0; d < HD; ++d) acc = fmaf(qs[i][d], kt[j][d], acc);
                    s = acc * scale;
                }
                sc[i][j] = s;
            }
            __syncthreads();
            if (tid < 16) {
                float mx = -INFINITY;
                for (int j = 0; j < DV_ATTN_TILE; ++j) mx = fmaxf(mx, sc[tid][j]);
                const float mold = mrun[tid];
                const float mnew = fmaxf(mold, mx);
                float al = 1.f, sum = 0.f;
                if (mnew != -INFINITY) {
                    al = (mold == -INFINITY) ? 0.f : expf(mold - mnew);
                    for (int j = 0; j < DV_ATTN_TILE; ++j) {
                        const float s = sc[tid][j];
                        const float p = (s == -INFINITY) ? 0.f : expf(s - mnew);
                        sc[tid][j] = p;
                        sum += p;
                    }
                } else {
                    for (int j = 0; j < DV_ATTN_TILE; ++j) sc[tid][j] = 0.f;
                }
                lrun[tid] = lrun[tid] * al + sum;
                mrun[tid] = mnew;
                alph[tid] = al;
            }
            __syncthreads();
            {
                const float al = alph[qi];
#pragma unroll
                for (int c = 0; c < DPT; ++c) {
                    float acc = o[c] * al;
                    for (int j = 0; j < DV_ATTN_TILE; ++j) acc = fmaf(sc[qi][j], vt[j][dd + c], acc);
                    o[c] = acc;
                }
            }
            __syncthreads();
        }
        const size_t pbase = ((size_t)h * a.n_split + split) * DV_TREE_MAX;
        if (qi < nq) {
#pragma unroll
            for (int c = 0; c < DPT; ++c) a.part_o[(pbase + q0 + qi) * HD + dd + c] = o[c];
        }
        if (tid < nq) {
            a.part_m[pbase + q0 + tid] = mrun[tid];
            a.part_l[pbase + q0 + tid] = lrun[tid];
        }
        __syncthreads();
    }
}

// Combine the splits of each (node, head): softmax-weighted sum of the split
// outputs in split order.  Grid (Mpad, H), block hd threads; rows >= M are 0.
__global__ void k_attn_merge(AttnArgs a)
{
    const int i = blockIdx.x, h = blockIdx.y, d = threadIdx.x, HD = a.hd;
    const int M = a.sd->M;
    float *out = a.out + (size_t)i * a.H * HD + h * HD + d;
    if (i >= M) { *out = 0.f; return; }
    const size_t base = (size_t)h * a.n_split * DV_TREE_MAX + i;
    float mx = -INFINITY;
    for (int s = 0; s < a.n_split; ++s) mx = fmaxf(mx, a.part_m[base + (size_t)s * DV_TREE_MAX]);
    float l = 0.f, o = 0.f;
    for (int s = 0; s < a.n_split; ++s) {
        const size_t ps = base + (size_t)s * DV_TREE_MAX;
        const float ms = a.part_m[ps];
        if (ms == -INFINITY) continue;
        const float w = expf(ms - mx);
        l = fmaf(w, a.part_l[ps], l);
        o = fmaf(w, a.part_o[ps * HD + d], o);
    }
    *out = o / l;
}

// ---------------------------------------------------------------------------
// Vocab-wide argmax and the greedy acceptance walk over the tree.
// 16 threads per node scan the per-tile (max, argmax) partials; the (value,
// index) pairs are combined by "larger value, then smaller index", which is
// order-independent, so ties resolve to the lowest token id.

__device__ __forceinline__ void arg_better(float &v, int &i, float v2, int i2)
{
    if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
}

__global__ __launch_bounds__(1024) void k_accept(AcceptArgs a)
{
    __shared__ int32_t amax[DV_TREE_MAX];
    __shared__ int32_t ok[DV_TREE_MAX];
    const StepDesc *sd = a.sd;
    const int M = sd->M, tid = threadIdx.x;
    const int m = tid >> 4, sub = tid & 15;
    if (m < M) {
        const float *val = a.arg_val + (size_t)m * a.n_tiles;
        const int32_t *idx = a.arg_idx + (size_t)m * a.n_tiles;
        float best = -INFINITY;
        int bi = 0x7fffffff;
        for (int t = sub; t < a.n_tiles; t += 16) arg_better(best, bi, val[t], idx[t]);
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) {
            const float v2 = __shfl_xor(best, off, 16);
            const int i2 = __shfl_xor(bi, off, 16);
            arg_better(best, bi, v2, i2);
        }
        if (sub == 0) {
            amax[m] = bi;
            a.acc->argmax[m] = bi;
        }
    }
    __syncthreads();
    if (tid == 0) {
        ok[0] = 1;
        int best = 0;
        for (int i = 1; i < M; ++i) {
            const int p = sd->parents[i];
            ok[i] = ok[p] && sd->tokens[i] == amax[p];
            if (ok[i] && sd->depth[i] > sd->depth[best]) best = i;
        }
        const int n = sd->depth[best];
        int node = best;
        for (int k = n - 1; k >= 0; --k) {
            a.acc->path[k] = node;
            node = sd->parents[node];
        }
        a.acc->accept_len = n;
        a.acc->bonus = amax[best];
    }
}

// ---------------------------------------------------------------------------
// KV commit: slot P+k <- slot P+path[k] for k < n, for every (layer, head)
// of K (blockIdx.y = 0) and V (1).  A destination can be the source of
// another k, so every row is read into LDS before any row is written.

template <typename KV>
__global__ __launch_bounds__(256) void k_kv_commit(CommitArgs a)
{
    __shared__ KV buf[DV_TREE_MAX * 128];
    KV *base = reinterpret_cast<KV *>(blockIdx.y ? a.vc : a.kc) + (size_t)blockIdx.x * a.cap * a.hd;
    const int nel = a.n * a.hd;
    for (int e = threadIdx.x; e < nel; e += blockDim.x) {
        const int k = e / a.hd, d = e % a.hd;
        buf[e] = base[(size_t)(a.P + a.path[k]) * a.hd + d];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < nel; e += blockDim.x) {
        const int k = e / a.hd, d = e % a.hd;
        if (a.path[k] != k) base[(size_t)(a.P + k) * a.hd + d] = buf[e];
    }
}

// ---------------------------------------------------------------------------
// launchers

template <int EPI, typename KV>
static const void *gemm_kernel(int weight_bf16, int use_mfma, int mt)
{
    if (weight_bf16 && use_mfma) {
        switch (mt) {
        case 1: return (const void *)k_gemm_mfma<1, EPI, KV>;
        case 2: return (const void *)k_gemm_mfma<2, EPI, KV>;
        case 3: return (const void *)k_gemm_mfma<3, EPI, KV>;
        case 4: return (const void *)k_gemm_mfma<4, EPI, KV>;
        default: return nullptr;
        }
    }
    if (weight_bf16) return (const void *)k_gemm_valu<uint16_t, EPI, KV>;
    return (const void *)k_gemm_valu<float, EPI, KV>;
}

static const void *gemm_kernel_any(int epi, int weight_bf16, int use_mfma, int mt)
{
    if (weight_bf16) {
        switch (epi) {
        case EPI_QKV: return gemm_kernel<EPI_QKV, uint16_t>(1, use_mfma, mt);
        case EPI_RESID: return gemm_kernel<EPI_RESID, uint16_t>(1, use_mfma, mt);
        case EPI_SWIGLU: return gemm_kernel<EPI_SWIGLU, uint16_t>(1, use_mfma, mt);
        case EPI_LOGITS: return gemm_kernel<EPI_LOGITS, uint16_t>(1, use_mfma, mt);
        }
    } else {
        switch (epi) {
        case EPI_QKV: return gemm_kernel<EPI_QKV, float>(0, 0, mt);
        case EPI_RESID: return gemm_kernel<EPI_RESID, float>(0, 0, mt);
        case EPI_SWIGLU: return gemm_kernel<EPI_SWIGLU, float>(0, 0, mt);
        case EPI_LOGITS: return gemm_kernel<EPI_LOGITS, float>(0, 0, mt);
        }
    }
    return nullptr;
}

hipError_t launch_pack(const GemmArgs &a, int epi, uint16_t *dst, hipStream_t s)
{
    hipLaunchKernelGGL(k_pack_tiles, dim3(a.n_tiles, std::min(a.K / 32, 64)), dim3(128), 0, s, a, epi, dst);
    return hipGetLastError();
}

int gemm_blocks_per_cu(int epi, int weight_bf16, int use_mfma, int mt)
{
    static int cache[4][2][2][5];
    int &c = cache[epi & 3][weight_bf16 ? 1 : 0][use_mfma ? 1 : 0][(mt >= 1 && mt <= 4) ? mt : 0];
    if (c == 0) {
        const void *k = gemm_kernel_any(epi, weight_bf16, use_mfma, mt);
        int n = 0;
        if (!k || hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, 256, 0) != hipSuccess || n < 1)
            n = 1;
        c = n;
    }
    return c;
}

hipError_t launch_gemm(const GemmArgs &a, int grid, int epi, int weight_bf16, int use_mfma,
                       hipStream_t s)
{
    const void *k = gemm_kernel_any(epi, weight_bf16, use_mfma, a.Mpad / 16);
    if (!k || grid < 1) return hipErrorInvalidValue;
    GemmArgs arg = a;
    void *params[] = {&arg};
    return hipLaunchKernel(k, dim3(grid), dim3(256), params, 0, s);
}

hipError_t launch_rmsnorm(const NormArgs &a, int Mpad, int weight_bf16, hipStream_t s)
{
    if (weight_bf16)
        hipLaunchKernelGGL(k_rmsnorm<uint16_t>, dim3(Mpad), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(k_rmsnorm<float>, dim3(Mpad), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs &a, int kv_bf16, hipStream_t s)
{
    const dim3 grid(a.n_split, a.H), block(256);
    if (a.hd == 128) {
        if (kv_bf16) hipLaunchKernelGGL((k_attn<128, uint16_t>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((k_attn<128, float>), grid, block, 0, s, a);
    } else if (a.hd == 64) {
        if (kv_bf16) hipLaunchKernelGGL((k_attn<64, uint16_t>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((k_attn<64, float>), grid, block, 0, s, a);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attn_merge(const AttnArgs &a, int Mpad, hipStream_t s)
{
    hipLaunchKernelGGL(k_attn_merge, dim3(Mpad, a.H), dim3(a.hd), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL(k_accept, dim3(1), dim3(1024), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_kv_commit(const CommitArgs &a, int kv_bf16, hipStream_t s)
{
    if (a.hd > 128) return hipErrorInvalidValue;
    if (kv_bf16)
        hipLaunchKernelGGL(k_kv_commit<uint16_t>, dim3(a.LH, 2), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(k_kv_commit<float>, dim3(a.LH, 2), dim3(256), 0, s, a);
    return hipGetLastError();
}
