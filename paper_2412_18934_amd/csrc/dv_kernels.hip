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
#include <hip/hip_ext.h>
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
// split layout of activations (see dv_internal.h)

__device__ __forceinline__ size_t split_index(int m, int k, int MT)
{
    const int s = k >> 5, g = (k >> 3) & 3, j = k & 7, mt = m >> 4, n = m & 15;
    return (((size_t)s * MT + mt) * 2 * 64 + g * 16 + n) * 8 + j;  // hi; lo is +512
}

__device__ __forceinline__ void store_split(uint16_t *xs, int m, int k, int MT, float v)
{
    const size_t i = split_index(m, k, MT);
    const float hi = __uint_as_float(__float_as_uint(v) & 0xffff0000u);
    xs[i] = (uint16_t)(__float_as_uint(v) >> 16);
    xs[i + 512] = f2bf(v - hi);
}

// fp32 -> bf16 hi (truncation) + lo (RNE of the remainder), 8 values
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

// four consecutive columns k..k+3 (k % 4 == 0) of one token
__device__ __forceinline__ void store_split4(uint16_t *xs, int m, int k, int MT, float4 v)
{
    const size_t i = split_index(m, k, MT);
    const float f[4] = {v.x, v.y, v.z, v.w};
    uint32_t hi[2], lo[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        uint32_t h2 = 0, l2 = 0;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const float x = f[2 * p + q];
            const float h = __uint_as_float(__float_as_uint(x) & 0xffff0000u);
            h2 |= (__float_as_uint(x) >> 16) << (16 * q);
            l2 |= (uint32_t)f2bf(x - h) << (16 * q);
        }
        hi[p] = h2;
        lo[p] = l2;
    }
    *reinterpret_cast<uint2 *>(xs + i) = make_uint2(hi[0], hi[1]);
    *reinterpret_cast<uint2 *>(xs + i + 512) = make_uint2(lo[0], lo[1]);
}

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
    if (EPI != EPI_RESID) {
        // 1/rms of each token (the normalisation the input skipped)
        __shared__ float rinv[DV_TREE_MAX];
        if (tid < a.Mpad) {
            float r = 0.f;
            if (tid < a.M) {
                float sq = 0.f;
#pragma unroll
                for (int sl = 0; sl < DV_NORM_SLICES; ++sl) sq += a.ssq[tid * DV_NORM_SLICES + sl];
                r = 1.0f / sqrtf(sq / (float)a.dn + a.eps);
            }
            rinv[tid] = r;
        }
        __syncthreads();
        for (int e = tid; e < a.Mpad * DV_GEMM_TILE; e += blockDim.x)
            tileY[e / DV_GEMM_TILE][e % DV_GEMM_TILE] *= rinv[e / DV_GEMM_TILE];
        __syncthreads();
    }
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
            const float hv = silu(tileY[m][r]) * tileY[m][16 + r];
            if (a.out_split) store_split(a.out_split, m, t * 16 + r, a.Mpad >> 4, hv);
            else a.out[(size_t)m * a.N + t * 16 + r] = hv;
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
            } else if (seg == 1) {  // K: [H][cap][hd]
                KV *c = reinterpret_cast<KV *>(a.kc);
                const size_t row = ((size_t)h * a.cap + a.P + m) * a.hd;
                Elem<KV>::store(c, row + j, y1);
                Elem<KV>::store(c, row + j + half, y2);
            } else {                // V: [H][hd][cap]
                KV *c = reinterpret_cast<KV *>(a.vc);
                const size_t col = (size_t)h * a.hd * a.cap + a.P + m;
                Elem<KV>::store(c, col + (size_t)j * a.cap, y1);
                Elem<KV>::store(c, col + (size_t)(j + half) * a.cap, y2);
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

#ifndef DV_WEIGHT_NT
#define DV_WEIGHT_NT 1
#endif
// Weights are read exactly once per step: the non-temporal hint keeps them
// from displacing reusable lines (activations) in the caches.
__device__ __forceinline__ u32x4 load_weights(const u32x4 *p)
{
    if (DV_WEIGHT_NT) return __builtin_nontemporal_load(p);
    return *p;
}

// N_STEPS k-steps for TP tiles: all weight and activation loads first, then
// the MFMAs (TP tiles x 2 halves x MT token tiles x hi/lo).
template <int MT, int TP, int N_STEPS>
__device__ __forceinline__ void mfma_steps(const uint16_t *wtile, size_t tile_stride,
                                           const uint16_t *xtile, f32x4 (&acc)[TP][2][MT])
{
    u32x4 wa[N_STEPS][TP][2];
    u32x4 xa[N_STEPS][MT][2];
#pragma unroll
    for (int u = 0; u < N_STEPS; ++u) {
#pragma unroll
        for (int p = 0; p < TP; ++p)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                wa[u][p][h] = load_weights(reinterpret_cast<const u32x4 *>(wtile + p * tile_stride + (2 * u + h) * 512));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int q = 0; q < 2; ++q)
                xa[u][mt][q] = *reinterpret_cast<const u32x4 *>(xtile + ((u * MT + mt) * 2 + q) * 512);
    }
#pragma unroll
    for (int u = 0; u < N_STEPS; ++u) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const bf16x8 hi = __builtin_bit_cast(bf16x8, xa[u][mt][0]);
            const bf16x8 lo = __builtin_bit_cast(bf16x8, xa[u][mt][1]);
#pragma unroll
            for (int p = 0; p < TP; ++p)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const bf16x8 w = __builtin_bit_cast(bf16x8, wa[u][p][h]);
                    acc[p][h][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, hi, acc[p][h][mt], 0, 0, 0);
                    acc[p][h][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, lo, acc[p][h][mt], 0, 0, 0);
                }
        }
    }
}

// MFMA GEMM for bf16 weights (packed tiles) and split-layout activations.
// v_mfma_f32_16x16x32_bf16: A = 16 weight rows x 32 k, B = 32 k x 16 tokens;
// each activation is the sum of its bf16 hi and lo parts, so every product
// keeps ~16 mantissa bits of the fp32 activation (two MFMAs per pair).
// D: lane l holds rows 4(l/16)..+4 of token l%16.
// Work unit = (TP consecutive tiles sharing the activation operand, K split).
// The grid is sized to stay resident and loops over units; within a unit the
// NW waves take contiguous shares of the k-steps, U k-steps per batch of
// loads, and their accumulators are summed in LDS in wave order.

template <int MT, int EPI, typename KV, int NW, int U, int TP>
__global__ __launch_bounds__(64 * NW) void k_gemm_mfma(GemmArgs a)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int K = a.K, S = K / 32;
    __shared__ float red[NW][2][MT][4][64];
    __shared__ float tileY[DV_TREE_MAX][TILE_LD];
    const int n_groups = a.n_tiles / TP;
    const size_t tile_stride = (size_t)S * 1024;

    for (int unit = blockIdx.x; unit < n_groups * a.ks; unit += gridDim.x) {
        const int tg = unit / a.ks, ksl = unit - tg * a.ks;
        const int sb = ksl * (a.k_per_split / 32);
        const int nsteps = min(S - sb, a.k_per_split / 32);
        const int s0 = sb + (wave * nsteps) / NW, s1 = sb + ((wave + 1) * nsteps) / NW;
        const uint16_t *wt = a.packed + (size_t)(tg * TP) * tile_stride + lane * 8;
        const uint16_t *xt = a.xs + lane * 8;

        f32x4 acc[TP][2][MT];
#pragma unroll
        for (int p = 0; p < TP; ++p)
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) acc[p][h][mt] = (f32x4){0.f, 0.f, 0.f, 0.f};
        int s = s0;
        for (; s + U <= s1; s += U)
            mfma_steps<MT, TP, U>(wt + (size_t)s * 1024, tile_stride, xt + (size_t)s * MT * 1024, acc);
        for (; s < s1; ++s)
            mfma_steps<MT, TP, 1>(wt + (size_t)s * 1024, tile_stride, xt + (size_t)s * MT * 1024, acc);

#pragma unroll
        for (int p = 0; p < TP; ++p) {
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int j = 0; j < 4; ++j) red[wave][h][mt][j][lane] = acc[p][h][mt][j];
            __syncthreads();
            for (int e = threadIdx.x; e < 2 * MT * 4 * 64; e += 64 * NW) {
                const int l = e & 63, j = (e >> 6) & 3, mt = (e >> 8) % MT, h = (e >> 8) / MT;
                float v = red[0][h][mt][j][l];
#pragma unroll
                for (int w = 1; w < NW; ++w) v += red[w][h][mt][j][l];
                tileY[mt * 16 + (l & 15)][h * 16 + 4 * (l >> 4) + j] = v;
            }
            __syncthreads();
            gemm_epilogue<EPI, KV>(a, tileY, tg * TP + p, ksl);
            __syncthreads();
        }
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

template <typename W, int NV, int KS>
__global__ __launch_bounds__(DV_NORM_THREADS) void k_rmsnorm(NormArgs a)
{
    constexpr int NT = DV_NORM_THREADS, SPAN = 4 * NT;
    const int m = blockIdx.x, sl = blockIdx.y, tid = threadIdx.x, d = a.d;
    const int c0 = sl * (d / DV_NORM_SLICES), c1 = c0 + d / DV_NORM_SLICES;
    float *urow = a.u + (size_t)m * d;
    float *xrow = a.x + (size_t)m * d;
    const int MT = gridDim.x >> 4;  // grid.x = Mpad rows
    if (m >= a.M) {
        for (int i = c0 + 4 * tid; i < c1; i += SPAN) {
            const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
            if (a.us) store_split4(a.us, m, i, MT, z);
            else *reinterpret_cast<float4 *>(urow + i) = z;
            if (a.embed) *reinterpret_cast<float4 *>(xrow + i) = z;
        }
        if (tid == 0) a.ssq[m * DV_NORM_SLICES + sl] = 0.f;
        return;
    }
    // NV = ceil(slice / SPAN) float4 per thread; KS = number of split-K
    // partials to add (compile-time, so that all loads of the slice are
    // issued together; KS < 0: a runtime count).  Addresses are clamped, not
    // branched on: lanes past the slice end re-read its last float4 and drop it.
    int idx[NV];
#pragma unroll
    for (int c = 0; c < NV; ++c) idx[c] = min(c0 + 4 * tid + SPAN * c, c1 - 4);
    float4 v[NV];
    if (a.embed) {
        const W *e = reinterpret_cast<const W *>(a.embed) + (size_t)a.tokens[m] * d;
#pragma unroll
        for (int c = 0; c < NV; ++c)
            v[c] = make_float4(Elem<W>::load(e, idx[c]), Elem<W>::load(e, idx[c] + 1),
                               Elem<W>::load(e, idx[c] + 2), Elem<W>::load(e, idx[c] + 3));
    } else {
#pragma unroll
        for (int c = 0; c < NV; ++c) v[c] = *reinterpret_cast<const float4 *>(xrow + idx[c]);
    }
    const int ks = KS >= 0 ? KS : a.ks;
    if (KS > 0) {
        float4 q[KS > 0 ? KS : 1][NV];
#pragma unroll
        for (int s = 0; s < (KS > 0 ? KS : 1); ++s)
#pragma unroll
            for (int c = 0; c < NV; ++c)
                q[s][c] = *reinterpret_cast<const float4 *>(a.part + ((size_t)s * DV_TREE_MAX + m) * d + idx[c]);
#pragma unroll
        for (int s = 0; s < (KS > 0 ? KS : 1); ++s)
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                v[c].x += q[s][c].x; v[c].y += q[s][c].y; v[c].z += q[s][c].z; v[c].w += q[s][c].w;
            }
    } else {
        for (int s = 0; s < ks; ++s) {
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                const float4 q = *reinterpret_cast<const float4 *>(a.part + ((size_t)s * DV_TREE_MAX + m) * d + idx[c]);
                v[c].x += q.x; v[c].y += q.y; v[c].z += q.z; v[c].w += q.w;
            }
        }
    }
    const W *gp = reinterpret_cast<const W *>(a.gain);
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NV; ++c) {
        const int i = idx[c];
        if (c0 + 4 * tid + SPAN * c < c1) {
            if (a.embed || ks) *reinterpret_cast<float4 *>(xrow + i) = v[c];
            ss = fmaf(v[c].x, v[c].x, ss);
            ss = fmaf(v[c].y, v[c].y, ss);
            ss = fmaf(v[c].z, v[c].z, ss);
            ss = fmaf(v[c].w, v[c].w, ss);
            float4 o;
            o.x = v[c].x * Elem<W>::load(gp, i);
            o.y = v[c].y * Elem<W>::load(gp, i + 1);
            o.z = v[c].z * Elem<W>::load(gp, i + 2);
            o.w = v[c].w * Elem<W>::load(gp, i + 3);
            if (a.us) store_split4(a.us, m, i, MT, o);
            else *reinterpret_cast<float4 *>(urow + i) = o;
        }
    }
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    __shared__ float wsum[NT / 64];
    if ((tid & 63) == 0) wsum[tid >> 6] = ss;
    __syncthreads();
    if (tid == 0) {
        float tot = 0.f;
#pragma unroll
        for (int w = 0; w < NT / 64; ++w) tot += wsum[w];
        a.ssq[m * DV_NORM_SLICES + sl] = tot;
    }
}

// ---------------------------------------------------------------------------
// Tree-masked attention, split over keys (flash-decoding style).
//
// Cache layouts: K [H][cap][hd] (key-major), V [H][hd][cap] (dim-major).
// Workgroup (split s, head h) covers keys [s*kps, (s+1)*kps) of the P + M
// cache slots; the tree's own keys/values were written to slots P.. by the
// QKV epilogue.  Key j is visible to node i iff j < P or bit (j-P) of
// anc(i).  Each split writes its unnormalised output with the running max
// and sum; k_attn_merge combines the splits (or, with one split, the
// workgroup writes the normalised output itself).

// bf16 cache, MFMA.  Queries are taken 16 at a time; the NW waves take
// interleaved 32-key tiles and are combined in LDS at the end.
//   S^T = K Q^T: A = 16 keys x 32 dims (16 bytes of one key row per lane),
//   B = Q^T (fp32 queries split into bf16 hi + lo, staged in LDS).  Tile "a"
//   holds keys k0 + 8(r/4) + r%4 in row r, tile "b" the same + 4, so lane l
//   ends up with the scores of token l%16 for the 8 consecutive keys
//   k0 + 8(l/16) .. +8.
//   O = P V: A = P (those 8 scores per lane, exponentiated, split hi + lo),
//   B = V^T rows: 16 bytes = the same 8 consecutive keys of one dim.
// Scores are kept in base-2 units (scaled by log2(e)/sqrt(hd)) so every
// exponential is one exp2; the running max written for the merge is
// converted back to natural units.  Each wave keeps two tiles of K and V in
// registers (the next one loads while the current one is used); the
// prologue issues the query, ancestor-mask and first-tile loads together.

template <int HD, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn_mfma(AttnArgs a)
{
    constexpr int NC = HD / 32;  // QK k-steps over dims
    constexpr int ND = HD / 16;  // PV output dim tiles
    static_assert(64 * NW >= 2 * HD, "one thread per 8 query values");
    const int split = blockIdx.x, h = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, g = lane >> 4;
    const StepDesc *sd = a.sd;
    const int M = sd->M, P = sd->P, total = P + M;
    const int kbeg = split * a.keys_per_split;
    const int kend = min(total, kbeg + a.keys_per_split);
    const int ntile = (kend - kbeg + 31) / 32;
    const int D = a.H * HD;
    const float scale2 = 1.4426950408889634f / sqrtf((float)HD);
    const uint16_t *kc = reinterpret_cast<const uint16_t *>(a.kc) + (size_t)h * a.cap * HD;
    const uint16_t *vc = reinterpret_cast<const uint16_t *>(a.vc) + (size_t)h * HD * a.cap;

    __shared__ u32x4 sm_q[NC * 2 * 64];  // [k-step][hi/lo][lane] B operands
    __shared__ float sm_m[NW][16], sm_l[NW][16];
    __shared__ float sm_o[NW][16][HD + 4];

    struct Tile {
        u32x4 ka[NC], kb[NC], v[ND];
    };
    auto load = [&](int t, Tile &T) {
        const int k0 = kbeg + 32 * t;
        const int ka = min(k0 + 8 * (n >> 2) + (n & 3), kend - 1);
        const int kb = min(k0 + 8 * (n >> 2) + 4 + (n & 3), kend - 1);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            T.ka[c] = *reinterpret_cast<const u32x4 *>(kc + (size_t)ka * HD + 32 * c + 8 * g);
            T.kb[c] = *reinterpret_cast<const u32x4 *>(kc + (size_t)kb * HD + 32 * c + 8 * g);
        }
        // columns past the last cache slot of the tile stay inside the
        // allocation (capacity is a multiple of 32); they are masked below
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
            T.v[dt] = *reinterpret_cast<const u32x4 *>(vc + (size_t)(dt * 16 + n) * a.cap + k0 + 8 * g);
    };

    for (int q0 = 0; q0 < M; q0 += 16) {
        const int tok = q0 + n;
        const bool tok_ok = tok < M;
        // thread e < 2*HD converts 8 dims (c, group qg) of query row qt
        const int e = threadIdx.x;
        const int qt = e / (2 * NC * 2) % 16, qc = (e >> 2) % NC, qg = e & 3;
        float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
        if (e < 2 * HD) {
            const float *qp = a.q + (size_t)min(q0 + qt, M - 1) * D + h * HD + qc * 32 + qg * 8;
            x0 = *reinterpret_cast<const float4 *>(qp);
            x1 = *reinterpret_cast<const float4 *>(qp + 4);
        }
        const uint64_t anc_raw = sd->anc[min(tok, M - 1)];
        Tile buf0, buf1;
        if (wave < ntile) load(wave, buf0);
        const uint64_t anc = tok_ok ? anc_raw : 0ull;
        if (e < 2 * HD) {
            const float qs = q0 + qt < M ? 1.f : 0.f;
            x0.x *= qs; x0.y *= qs; x0.z *= qs; x0.w *= qs;
            x1.x *= qs; x1.y *= qs; x1.z *= qs; x1.w *= qs;
            bf16x8 hh, ll;
            split_hi_lo(x0, x1, hh, ll);
            sm_q[(qc * 2 + 0) * 64 + 16 * qg + qt] = __builtin_bit_cast(u32x4, hh);
            sm_q[(qc * 2 + 1) * 64 + 16 * qg + qt] = __builtin_bit_cast(u32x4, ll);
        }
        __syncthreads();

        float m_run = -INFINITY, l_run = 0.f;
        f32x4 o[ND];
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) o[dt] = (f32x4){0.f, 0.f, 0.f, 0.f};

        auto process = [&](int t, Tile &cur) {
            const int k0 = kbeg + 32 * t;
            f32x4 sa = (f32x4){0.f, 0.f, 0.f, 0.f}, sb = sa;
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const bf16x8 ka8 = __builtin_bit_cast(bf16x8, cur.ka[c]);
                const bf16x8 kb8 = __builtin_bit_cast(bf16x8, cur.kb[c]);
                const bf16x8 qh = __builtin_bit_cast(bf16x8, sm_q[(c * 2 + 0) * 64 + lane]);
                const bf16x8 ql = __builtin_bit_cast(bf16x8, sm_q[(c * 2 + 1) * 64 + lane]);
                sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka8, qh, sa, 0, 0, 0);
                sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb8, qh, sb, 0, 0, 0);
                sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka8, ql, sa, 0, 0, 0);
                sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb8, ql, sb, 0, 0, 0);
            }
            float sv[8];
            float mt = -INFINITY;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int key = k0 + 8 * g + i;
                const int sh = key - P;
                const bool tree_ok = sh < 0 || ((anc >> (sh & 63)) & 1ull);
                const bool vis = key < kend && tree_ok;
                const float sc = (i < 4 ? sa[i] : sb[i - 4]) * scale2;
                sv[i] = vis ? sc : -INFINITY;
                mt = fmaxf(mt, sv[i]);
            }
            mt = fmaxf(mt, __shfl_xor(mt, 16));
            mt = fmaxf(mt, __shfl_xor(mt, 32));
            const float mnew = fmaxf(m_run, mt);
            const float alpha = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - mnew);
            float ps = 0.f, pv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                pv[i] = sv[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sv[i] - mnew);
                ps += pv[i];
            }
            ps += __shfl_xor(ps, 16);
            ps += __shfl_xor(ps, 32);
            l_run = l_run * alpha + ps;
            m_run = mnew;
            // O rows held by this lane are tokens 4g + j
            float al[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) al[j] = __shfl(alpha, 4 * g + j);
            if (k0 + 32 > kend) {
                // ragged last tile: values of slots past the split end are dropped
#pragma unroll
                for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const int key = k0 + 8 * g + 2 * w;
                        uint32_t x = cur.v[dt][w];
                        if (key >= kend) x &= 0xffff0000u;
                        if (key + 1 >= kend) x &= 0x0000ffffu;
                        cur.v[dt][w] = x;
                    }
            }
            bf16x8 ph, pl;
            split_hi_lo(make_float4(pv[0], pv[1], pv[2], pv[3]), make_float4(pv[4], pv[5], pv[6], pv[7]), ph, pl);
#pragma unroll
            for (int dt = 0; dt < ND; ++dt) {
#pragma unroll
                for (int j = 0; j < 4; ++j) o[dt][j] *= al[j];
                const bf16x8 v8 = __builtin_bit_cast(bf16x8, cur.v[dt]);
                o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, v8, o[dt], 0, 0, 0);
                o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, v8, o[dt], 0, 0, 0);
            }
        };
        // two register buffers used in turn (no copies between them, so a
        // load in flight is never waited on before its tile is used)
        for (int t = wave; t < ntile; t += 2 * NW) {
            if (t + NW < ntile) load(t + NW, buf1);
            process(t, buf0);
            if (t + NW >= ntile) break;
            if (t + 2 * NW < ntile) load(t + 2 * NW, buf0);
            process(t + NW, buf1);
        }

        // combine the waves (fixed wave order)
        if (g == 0) {
            sm_m[wave][n] = m_run;
            sm_l[wave][n] = l_run;
        }
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
#pragma unroll
            for (int j = 0; j < 4; ++j) sm_o[wave][4 * g + j][dt * 16 + n] = o[dt][j];
        __syncthreads();
        for (int e2 = threadIdx.x; e2 < 16 * HD; e2 += 64 * NW) {
            const int i = e2 / HD, dd = e2 % HD;
            const int ti = q0 + i;
            float mx = -INFINITY;
#pragma unroll
            for (int w = 0; w < NW; ++w) mx = fmaxf(mx, sm_m[w][i]);
            float l = 0.f, ov = 0.f;
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const float mw = sm_m[w][i];
                const float wgt = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - mx);
                l = fmaf(wgt, sm_l[w][i], l);
                ov = fmaf(wgt, sm_o[w][i][dd], ov);
            }
            if (a.n_split == 1) {
                if (ti < sd->Mpad) {
                    const float r = ti < M ? ov / l : 0.f;
                    if (a.out_split) store_split(a.out_split, ti, h * HD + dd, sd->Mpad >> 4, r);
                    else a.out[(size_t)ti * D + h * HD + dd] = r;
                }
            } else if (ti < M) {
                const size_t pb = ((size_t)h * a.n_split + split) * DV_TREE_MAX + ti;
                a.part_o[pb * HD + dd] = ov;
                if (dd == 0) {
                    a.part_m[pb] = mx * 0.6931471805599453f;  // back to natural-log units
                    a.part_l[pb] = l;
                }
            }
        }
        __syncthreads();
    }
}

// fp32 cache (VALU).  K/V tiles of 32 keys sit in LDS as fp32; 16 queries
// at a time; an online softmax keeps (max, sum, o) per query.

template <int HD>
__global__ __launch_bounds__(256) void k_attn_f32(AttnArgs a)
{
    constexpr int DPT = HD / 16;  // output dims per thread
    const int split = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const StepDesc *sd = a.sd;
    const int M = sd->M, P = sd->P, total = P + M;
    const int kb = split * a.keys_per_split;
    const int ke = min(total, kb + a.keys_per_split);
    const float scale = 1.0f / sqrtf((float)HD);
    const float *kc = reinterpret_cast<const float *>(a.kc) + (size_t)h * a.cap * HD;
    const float *vc = reinterpret_cast<const float *>(a.vc) + (size_t)h * HD * a.cap;
    const int D = a.H * HD;

    __shared__ float qs[16][HD];
    __shared__ float kt[DV_ATTN_TILE][HD + 1];
    __shared__ float vt[DV_ATTN_TILE][HD + 1];
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
                kt[j][d] = j < nk ? kc[(size_t)(t0 + j) * HD + d] : 0.f;
                const int jv = e % DV_ATTN_TILE, dv = e / DV_ATTN_TILE;
                vt[jv][dv] = jv < nk ? vc[(size_t)dv * a.cap + t0 + jv] : 0.f;
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
                        const float sj = sc[tid][j];
                        const float p = (sj == -INFINITY) ? 0.f : expf(sj - mnew);
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
        if (a.n_split == 1) {
            if (q0 + qi < sd->Mpad) {
#pragma unroll
                for (int c = 0; c < DPT; ++c) {
                    const float r = qi < nq ? o[c] / lrun[qi] : 0.f;
                    if (a.out_split) store_split(a.out_split, q0 + qi, h * HD + dd + c, sd->Mpad >> 4, r);
                    else a.out[(size_t)(q0 + qi) * D + h * HD + dd + c] = r;
                }
            }
        } else {
            const size_t pbase = ((size_t)h * a.n_split + split) * DV_TREE_MAX;
            if (qi < nq) {
#pragma unroll
                for (int c = 0; c < DPT; ++c) a.part_o[(pbase + q0 + qi) * HD + dd + c] = o[c];
            }
            if (tid < nq) {
                a.part_m[pbase + q0 + tid] = mrun[tid];
                a.part_l[pbase + q0 + tid] = lrun[tid];
            }
        }
        __syncthreads();
    }
}

// Combine the splits of each (node, head): softmax-weighted sum of the split
// outputs.  Splits are read 16 at a time (all loads of a chunk in flight
// together) and folded in split order with a running maximum.  Grid (Mpad, H),
// block hd threads; rows >= M are 0.
__global__ __launch_bounds__(128) void k_attn_merge(AttnArgs a)
{
    constexpr int CH = 16;
    const int i = blockIdx.x, h = blockIdx.y, d = threadIdx.x, HD = a.hd;
    const int M = a.sd->M, MT = gridDim.x >> 4;
    if (i >= M) {
        if (a.out_split) store_split(a.out_split, i, h * HD + d, MT, 0.f);
        else a.out[(size_t)i * a.H * HD + h * HD + d] = 0.f;
        return;
    }
    const size_t base = (size_t)h * a.n_split * DV_TREE_MAX + i;
    float run_m = -INFINITY, l = 0.f, o = 0.f;
    for (int s0 = 0; s0 < a.n_split; s0 += CH) {
        float ms[CH], ls[CH], os[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const size_t ps = base + (size_t)min(s0 + c, a.n_split - 1) * DV_TREE_MAX;
            ms[c] = a.part_m[ps];
            ls[c] = a.part_l[ps];
            os[c] = a.part_o[ps * HD + d];
        }
        float mx = run_m;
#pragma unroll
        for (int c = 0; c < CH; ++c)
            if (s0 + c < a.n_split) mx = fmaxf(mx, ms[c]);
        if (mx == -INFINITY) continue;
        const float sc = run_m == -INFINITY ? 0.f : expf(run_m - mx);
        l *= sc;
        o *= sc;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            if (s0 + c < a.n_split && ms[c] != -INFINITY) {
                const float w = expf(ms[c] - mx);
                l = fmaf(w, ls[c], l);
                o = fmaf(w, os[c], o);
            }
        }
        run_m = mx;
    }
    if (a.out_split) store_split(a.out_split, i, h * HD + d, MT, o / l);
    else a.out[(size_t)i * a.H * HD + h * HD + d] = o / l;
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
    // tpt threads per node (64, 32 or 16), each scanning a contiguous chunk of
    // the tiles 16 loads at a time (clamped indices only repeat a real entry)
    const int tpt = sd->Mpad <= 16 ? 64 : (sd->Mpad <= 32 ? 32 : 16);
    const int m = tid / tpt, sub = tid % tpt;
    if (m < M) {
        const float *val = a.arg_val + (size_t)m * a.n_tiles;
        const int32_t *idx = a.arg_idx + (size_t)m * a.n_tiles;
        const int chunk = (a.n_tiles + tpt - 1) / tpt;
        const int t0 = sub * chunk, t1 = min(a.n_tiles, t0 + chunk);
        float best = -INFINITY;
        int bi = 0x7fffffff;
        for (int t = t0; t < t1; t += 16) {
            float v[16];
            int ix[16];
#pragma unroll
            for (int c = 0; c < 16; ++c) {
                const int tt = min(t + c, t1 - 1);
                v[c] = val[tt];
                ix[c] = idx[tt];
            }
#pragma unroll
            for (int c = 0; c < 16; ++c) arg_better(best, bi, v[c], ix[c]);
        }
        for (int off = tpt >> 1; off > 0; off >>= 1) {
            const float v2 = __shfl_xor(best, off, tpt);
            const int i2 = __shfl_xor(bi, off, tpt);
            arg_better(best, bi, v2, i2);
        }
        if (sub == 0) {
            amax[m] = bi;
            a.acc->argmax[m] = bi;
        }
    }
    // the tree in LDS, so the serial walk below makes no global round trips
    __shared__ int32_t par_s[DV_TREE_MAX], tok_s[DV_TREE_MAX], dep_s[DV_TREE_MAX];
    if (tid < M) {
        par_s[tid] = sd->parents[tid];
        tok_s[tid] = sd->tokens[tid];
        dep_s[tid] = sd->depth[tid];
    }
    __syncthreads();
    if (tid == 0) {
        ok[0] = 1;
        int best = 0;
        for (int i = 1; i < M; ++i) {
            const int p = par_s[i];
            ok[i] = ok[p] && tok_s[i] == amax[p];
            if (ok[i] && dep_s[i] > dep_s[best]) best = i;
        }
        const int n = dep_s[best];
        int node = best;
        for (int k = n - 1; k >= 0; --k) {
            a.acc->path[k] = node;
            node = par_s[node];
        }
        a.acc->accept_len = n;
        a.acc->bonus = amax[best];
    }
}

// ---------------------------------------------------------------------------
// KV commit: slot P+k <- slot P+path[k] for k < n, for every (layer, head)
// of K (blockIdx.y = 0, rows [cap][hd]) and V (1, columns of [hd][cap]).  A
// destination can be the source of another k, so every entry is read into
// LDS before any entry is written.

template <typename KV>
__global__ __launch_bounds__(256) void k_kv_commit(CommitArgs a)
{
    __shared__ KV buf[DV_TREE_MAX * 128];
    const bool is_v = blockIdx.y != 0;
    KV *base = reinterpret_cast<KV *>(is_v ? a.vc : a.kc) + (size_t)blockIdx.x * a.cap * a.hd;
    const int nel = a.n * a.hd;
    for (int e = threadIdx.x; e < nel; e += blockDim.x) {
        const int k = e / a.hd, d = e % a.hd;
        const size_t src = is_v ? (size_t)d * a.cap + a.P + a.path[k] : (size_t)(a.P + a.path[k]) * a.hd + d;
        buf[e] = base[src];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < nel; e += blockDim.x) {
        const int k = e / a.hd, d = e % a.hd;
        if (a.path[k] == k) continue;
        const size_t dst = is_v ? (size_t)d * a.cap + a.P + k : (size_t)(a.P + k) * a.hd + d;
        base[dst] = buf[e];
    }
}

// ---------------------------------------------------------------------------
// launchers

// Load batch per variant: U k-steps for one token tile, fewer as MT grows
// (register budget); waves per workgroup capped at 4 for MT >= 3.
template <int EPI, typename KV, int NW, int U, int TP>
static const void *gemm_kernel_mfma(int mt)
{
    // more token tiles hold more accumulators: fewer k-steps per batch
    switch (mt) {
    case 1: return (const void *)k_gemm_mfma<1, EPI, KV, NW, U, TP>;
    case 2: return (const void *)k_gemm_mfma<2, EPI, KV, NW, (U > 4 ? U / 2 : 2), TP>;
    case 3: return (const void *)k_gemm_mfma<3, EPI, KV, 4, 2, TP>;
    case 4: return (const void *)k_gemm_mfma<4, EPI, KV, 4, (TP > 2 ? 1 : 2), TP>;
    default: return nullptr;
    }
}

// index of an instantiated shape, -1 if none
static int shape_index(GemmShape sh)
{
    if (sh.nw == 8 && sh.u == 4 && sh.tp == 2) return 0;
    if (sh.nw == 4 && sh.u == 8 && sh.tp == 2) return 1;
    if (sh.nw == 4 && sh.u == 4 && sh.tp == 4) return 2;
    if (sh.nw == 4 && sh.u == 8 && sh.tp == 1) return 3;
    return -1;
}

template <int EPI>
static const void *gemm_kernel(int weight_bf16, int use_mfma, int mt, GemmShape sh)
{
    if (weight_bf16 && use_mfma) {
        switch (shape_index(sh)) {
        case 0: return gemm_kernel_mfma<EPI, uint16_t, 8, 4, 2>(mt);
        case 1: return gemm_kernel_mfma<EPI, uint16_t, 4, 8, 2>(mt);
        case 2: return gemm_kernel_mfma<EPI, uint16_t, 4, 4, 4>(mt);
        case 3: return gemm_kernel_mfma<EPI, uint16_t, 4, 8, 1>(mt);
        default: return nullptr;
        }
    }
    if (weight_bf16) return (const void *)k_gemm_valu<uint16_t, EPI, uint16_t>;
    return (const void *)k_gemm_valu<float, EPI, float>;
}

static const void *gemm_kernel_any(int epi, int weight_bf16, int use_mfma, int mt, GemmShape sh)
{
    switch (epi) {
    case EPI_QKV: return gemm_kernel<EPI_QKV>(weight_bf16, use_mfma, mt, sh);
    case EPI_RESID: return gemm_kernel<EPI_RESID>(weight_bf16, use_mfma, mt, sh);
    case EPI_SWIGLU: return gemm_kernel<EPI_SWIGLU>(weight_bf16, use_mfma, mt, sh);
    case EPI_LOGITS: return gemm_kernel<EPI_LOGITS>(weight_bf16, use_mfma, mt, sh);
    }
    return nullptr;
}

static int gemm_threads(int weight_bf16, int use_mfma, int mt, GemmShape sh)
{
    if (!(weight_bf16 && use_mfma)) return 256;
    return mt >= 3 ? 256 : 64 * sh.nw;
}

int gemm_blocks_per_cu(int epi, int weight_bf16, int use_mfma, int mt, GemmShape sh)
{
    static int cache[4][2][2][5][5];
    int &c = cache[epi & 3][weight_bf16 ? 1 : 0][use_mfma ? 1 : 0][(mt >= 1 && mt <= 4) ? mt : 0]
                  [shape_index(sh) + 1];
    if (c == 0) {
        const void *k = gemm_kernel_any(epi, weight_bf16, use_mfma, mt, sh);
        int n = 0;
        if (!k || hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, gemm_threads(weight_bf16, use_mfma, mt, sh),
                                                               0) != hipSuccess || n < 1)
            n = 1;
        c = n;
    }
    return c;
}

hipError_t launch_gemm(const GemmArgs &a, int grid, int epi, int weight_bf16, int use_mfma,
                       GemmShape sh, hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop)
{
    const void *k = gemm_kernel_any(epi, weight_bf16, use_mfma, a.Mpad / 16, sh);
    if (!k || grid < 1) return hipErrorInvalidValue;
    GemmArgs arg = a;
    void *params[] = {&arg};
    const dim3 block(gemm_threads(weight_bf16, use_mfma, a.Mpad / 16, sh));
    // with events: timestamps taken by the dispatch itself (no extra packets)
    if (ev_start && ev_stop) return hipExtLaunchKernel(k, dim3(grid), block, params, 0, s, ev_start, ev_stop, 0);
    return hipLaunchKernel(k, dim3(grid), block, params, 0, s);
}

hipError_t launch_pack(const GemmArgs &a, int epi, uint16_t *dst, hipStream_t s)
{
    hipLaunchKernelGGL(k_pack_tiles, dim3(a.n_tiles, std::min(a.K / 32, 64)), dim3(128), 0, s, a, epi, dst);
    return hipGetLastError();
}

template <typename W, int NV>
static hipError_t rmsnorm_dispatch_ks(const NormArgs &a, int Mpad, hipStream_t s)
{
    const dim3 grid(Mpad, DV_NORM_SLICES), block(DV_NORM_THREADS);
    switch (a.ks) {
    case 0: hipLaunchKernelGGL((k_rmsnorm<W, NV, 0>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_rmsnorm<W, NV, 2>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_rmsnorm<W, NV, 4>), grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_rmsnorm<W, NV, 8>), grid, block, 0, s, a); break;
    case 16: hipLaunchKernelGGL((k_rmsnorm<W, NV, 16>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((k_rmsnorm<W, NV, -1>), grid, block, 0, s, a); break;
    }
    return hipGetLastError();
}

template <typename W>
static hipError_t rmsnorm_dispatch(const NormArgs &a, int Mpad, hipStream_t s)
{
    const int slice = a.d / DV_NORM_SLICES;
    if (a.d % (4 * DV_NORM_SLICES)) return hipErrorInvalidValue;
    switch ((slice + 4 * DV_NORM_THREADS - 1) / (4 * DV_NORM_THREADS)) {
    case 1: return rmsnorm_dispatch_ks<W, 1>(a, Mpad, s);
    case 2: return rmsnorm_dispatch_ks<W, 2>(a, Mpad, s);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_rmsnorm(const NormArgs &a, int Mpad, int weight_bf16, hipStream_t s)
{
    return weight_bf16 ? rmsnorm_dispatch<uint16_t>(a, Mpad, s) : rmsnorm_dispatch<float>(a, Mpad, s);
}

hipError_t launch_attention(const AttnArgs &a, int kv_bf16, hipStream_t s)
{
    const dim3 grid(a.n_split, a.H), block(256);
    const dim3 block8(64 * DV_ATTN_WAVES);
    if (a.hd == 128) {
        if (kv_bf16) hipLaunchKernelGGL((k_attn_mfma<128, DV_ATTN_WAVES>), grid, block8, 0, s, a);
        else hipLaunchKernelGGL(k_attn_f32<128>, grid, block, 0, s, a);
    } else if (a.hd == 64) {
        if (kv_bf16) hipLaunchKernelGGL((k_attn_mfma<64, DV_ATTN_WAVES>), grid, block8, 0, s, a);
        else hipLaunchKernelGGL(k_attn_f32<64>, grid, block, 0, s, a);
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
