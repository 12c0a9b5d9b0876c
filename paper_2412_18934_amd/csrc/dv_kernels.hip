// HIP kernels (gfx950 / CDNA4) for one tree-verification step.
//
// Step structure (Section 3.1 of the paper: one forward pass of the target
// over the candidate tokens, then the acceptance rule):
//   k_embed_norm     embedding gather + the first RMSNorm
//   k_proj / k_gemm_valu  weight-streaming projections with fused epilogues:
//                      QKV    -> 1/rms, rotary embedding, q store, K/V cache write
//                      RESID  -> residual add into the fp32 stream (O, down)
//                                and the next RMSNorm's x * gain and sums of squares
//                      SWIGLU -> 1/rms, silu(gate) * up
//                      LOGITS -> 1/rms, logits + per-group argmax
//   k_attn / merge   tree-masked attention over the cache, split over keys
//   k_accept         vocab-wide argmax reduce + greedy acceptance walk
//   k_accept_sampled speculative sampling walk over full logits rows (T > 0)
//   k_kv_commit      in-place compaction of the accepted path
//
// Weights are bf16 or fp32, activations and accumulation fp32.  Every
// reduction runs in a fixed order, so results are bitwise reproducible.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "dv.h"
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

// Buffer resource over a device allocation (byte offsets below 2 GiB) and the
// cache-policy bit of buffer instructions for data read once (non-temporal).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_of(const void *base)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, 0x7fffffff, 0x00020000);
}
#define DV_NT 2

// ---------------------------------------------------------------------------
// V cache layout: per (layer, head), 32-slot tiles one after another, each
// tile dim-major ([hd][32]): entry (dim j, slot s) at element
// ((s / 32) hd + j) 32 + s % 32 of the head, so one tile of 32 keys is one
// contiguous hd x 64-byte block and 8 consecutive slots of a dim are 16
// contiguous bytes (the PV B-operand).

__device__ __forceinline__ size_t v_index(int j, int s, int hd)
{
    return ((size_t)(s >> 5) * hd + j) * 32 + (s & 31);
}

// ---------------------------------------------------------------------------
// split layout of activations (see dv_internal.h)

// MT = 0 selects the half layout (tokens 0-7 only; lo in columns 8-15).
__device__ __forceinline__ size_t split_index(int m, int k, int MT)
{
    const int s = k >> 5, g = (k >> 3) & 3, j = k & 7, mt = m >> 4, n = m & 15;
    const size_t blk = MT ? ((size_t)s * MT + mt) * 2 : (size_t)s;
    return (blk * 64 + g * 16 + n) * 8 + j;  // hi; lo is + split_lo(MT)
}

__device__ __forceinline__ int split_lo(int MT) { return MT ? 512 : 64; }

// token tiles of a split-layout operand (0: half layout) and the tokens it
// holds
__device__ __forceinline__ int split_mt(int Mpad, int half) { return half ? 0 : Mpad >> 4; }
__device__ __forceinline__ int split_rows(int Mpad, int half) { return half ? 8 : Mpad; }

__device__ __forceinline__ void store_split(uint16_t *xs, int m, int k, int MT, float v)
{
    const size_t i = split_index(m, k, MT);
    const float hi = __uint_as_float(__float_as_uint(v) & 0xffff0000u);
    xs[i] = (uint16_t)(__float_as_uint(v) >> 16);
    xs[i + split_lo(MT)] = f2bf(v - hi);
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
    *reinterpret_cast<uint2 *>(xs + i + split_lo(MT)) = make_uint2(lo[0], lo[1]);
}

// ---------------------------------------------------------------------------
// Projection rows.  A 32-row tile is two 16-row halves (MFMA blocks) mapped to
// physical rows so that each epilogue finds the pair of values it needs in
// the same tile (see GemmArgs in dv_internal.h).

struct RowMap {
    const void *ptr[2];
    int32_t row0[2];
    int32_t mat[2];  // which of w0, w1, w2 each half reads
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
        m.mat[0] = m.mat[1] = seg;
        m.row0[0] = h * a.hd + j0;
        m.row0[1] = h * a.hd + a.hd / 2 + j0;
    } else if (epi == EPI_SWIGLU) {
        m.ptr[0] = a.w0;
        m.ptr[1] = a.w1;
        m.mat[0] = 0;
        m.mat[1] = 1;
        m.row0[0] = m.row0[1] = t * 16;
    } else {
        m.ptr[0] = m.ptr[1] = a.w0;
        m.mat[0] = m.mat[1] = 0;
        m.row0[0] = t * DV_GEMM_TILE;
        m.row0[1] = t * DV_GEMM_TILE + 16;
    }
    return m;
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// ---------------------------------------------------------------------------
// Projection epilogues.  Y[m * ld + r] (m < Mpad, r < rows) holds the
// complete sums of one row group's rows for token m.

// 1/rms of each token of the input from the producer's partial sums of
// squares, in a fixed order: thread 4 m + c sums partials c, c + 4, ...
// (loads issued together), then the four chains are combined by shuffles.
// Needs 4 Mpad <= blockDim.x; writes rinv[0..Mpad).
__device__ __forceinline__ void input_rinv(const GemmArgs &a, float *rinv)
{
    constexpr int NJ = 32;  // loads in flight per thread
    const int tid = threadIdx.x, m = tid >> 2, c = tid & 3;
    float s = 0.f;
    if (m < a.Mpad) {
        const float *p = a.ssq_in + (size_t)m * a.n_ssq_in;
        for (int base = 0; base < a.n_ssq_in; base += 4 * NJ) {
            float v[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const int i = base + c + 4 * j;
                v[j] = i < a.n_ssq_in ? p[i] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < NJ; ++j) s += v[j];
        }
    }
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    if (m < a.Mpad && c == 0) rinv[m] = m < a.M ? 1.0f / sqrtf(s / (float)a.dn + a.eps) : 0.f;
}

// The same 1/rms in two parts, for the projections: rinv_load issues the
// first NJ partials of each thread before the weight stream starts (loads
// return in order, so they arrive first and no later wait on them drains the
// stream); rinv_finish, after the stream, adds the remaining partials in the
// same order and writes rinv (bit-identical to input_rinv).
template <int NJ>
__device__ __forceinline__ void rinv_load(const GemmArgs &a, float (&v)[NJ])
{
    const int tid = threadIdx.x, m = tid >> 2, c = tid & 3;
    const float *p = a.ssq_in + (size_t)m * a.n_ssq_in;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int i = c + 4 * j;
        v[j] = (m < a.Mpad && i < a.n_ssq_in) ? p[i] : 0.f;
    }
}

template <int NJ>
__device__ __forceinline__ void rinv_finish(const GemmArgs &a, const float (&v)[NJ], float *rinv)
{
    const int tid = threadIdx.x, m = tid >> 2, c = tid & 3;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) s += v[j];
    if (m < a.Mpad) {
        const float *p = a.ssq_in + (size_t)m * a.n_ssq_in;
        for (int i = c + 4 * NJ; i < a.n_ssq_in; i += 4) s += p[i];
    }
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    if (m < a.Mpad && c == 0) rinv[m] = m < a.M ? 1.0f / sqrtf(s / (float)a.dn + a.eps) : 0.f;
}

// Residual projections: x += sums, then the next RMSNorm's numerator
// u = x * gain (split layout or fp32) and the group's sums of squares.
// Rows [row0, row0 + nrows) of the stream.  With y_is_x, Y already holds the
// updated rows x + sums and gain_s the gains of the rows (both staged in LDS
// by the caller); otherwise Y holds the sums and both are read here.  Y ends
// up holding x.
template <typename W>
__device__ void resid_epilogue(const GemmArgs &a, float *Y, int ld, int row0, int nrows, int group, bool y_is_x,
                               const float *gain_s)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    const W *gp = reinterpret_cast<const W *>(a.gain);
    for (int e = tid; e < a.Mpad * nrows; e += nt) {
        const int m = e / nrows, r = e - m * nrows;
        float v = 0.f;
        if (m < a.M) {
            float *xp = a.resid + (size_t)m * a.N + row0 + r;
            v = y_is_x ? Y[m * ld + r] : *xp + Y[m * ld + r];
            *xp = v;
        }
        Y[m * ld + r] = v;
    }
    __syncthreads();
    auto gain = [&](int r) -> float { return gain_s ? gain_s[r] : Elem<W>::load(gp, row0 + r); };
    if (a.us) {
        // 8 consecutive rows of one token per thread: one 16-byte hi and lo store
        const int MT = split_mt(a.Mpad, a.half), nc = nrows >> 3;
        for (int e = tid; e < split_rows(a.Mpad, a.half) * nc; e += nt) {
            const int m = e / nc, c = e - m * nc;
            const float *y = Y + m * ld + 8 * c;
            const int r = 8 * c;
            const float4 v0 = make_float4(y[0] * gain(r), y[1] * gain(r + 1), y[2] * gain(r + 2), y[3] * gain(r + 3));
            const float4 v1 = make_float4(y[4] * gain(r + 4), y[5] * gain(r + 5), y[6] * gain(r + 6), y[7] * gain(r + 7));
            bf16x8 hi, lo;
            split_hi_lo(v0, v1, hi, lo);
            const size_t i = split_index(m, row0 + r, MT);
            *reinterpret_cast<bf16x8 *>(a.us + i) = hi;
            *reinterpret_cast<bf16x8 *>(a.us + i + split_lo(MT)) = lo;
        }
    } else {
        for (int e = tid; e < a.Mpad * nrows; e += nt) {
            const int m = e / nrows, r = e - m * nrows;
            a.u[(size_t)m * a.N + row0 + r] = Y[m * ld + r] * gain(r);
        }
    }
    // sums of squares: 4 threads per token, fixed order
    if (tid < 4 * a.Mpad) {
        const int m = tid >> 2, c = tid & 3;
        float s = 0.f;
        for (int r = c; r < nrows; r += 4) s = fmaf(Y[m * ld + r], Y[m * ld + r], s);
        s += __shfl_xor(s, 1);
        s += __shfl_xor(s, 2);
        if (c == 0) a.ssq_out[(size_t)m * a.n_groups + group] = s;
    }
}

// The same for the MFMA projections' split-layout output, in one pass: each
// thread takes 8 consecutive rows of one token (Y already holds x + sums and
// gain_s the rows' gains), writes them to the stream, writes x * gain as one
// 16-byte hi and one lo store, and the 8 threads of a token sum their squares
// (each over its 8 rows in order, then combined by lane shuffles).
__device__ void resid_epilogue_split(const GemmArgs &a, const float *Y, int ld, int row0, int nrows, int group,
                                     const float *gain_s)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    const int MT = split_mt(a.Mpad, a.half), nc = nrows >> 3;  // chunks per token: 8 (64 rows) or 4 (32)
    const int total = split_rows(a.Mpad, a.half) * nc;
    for (int e0 = 0; e0 < total; e0 += nt) {
        const int e = e0 + tid;
        float s = 0.f;
        if (e < total) {
            const int m = e / nc, c = e - m * nc, r = 8 * c;
            const float *y = Y + m * ld + r;
            float4 v0 = make_float4(y[0], y[1], y[2], y[3]), v1 = make_float4(y[4], y[5], y[6], y[7]);
            if (m < a.M) {
                float *xp = a.resid + (size_t)m * a.N + row0 + r;
                *reinterpret_cast<float4 *>(xp) = v0;
                *reinterpret_cast<float4 *>(xp + 4) = v1;
            } else {
                v0 = v1 = make_float4(0.f, 0.f, 0.f, 0.f);
            }
            s = fmaf(v0.x, v0.x, s); s = fmaf(v0.y, v0.y, s); s = fmaf(v0.z, v0.z, s); s = fmaf(v0.w, v0.w, s);
            s = fmaf(v1.x, v1.x, s); s = fmaf(v1.y, v1.y, s); s = fmaf(v1.z, v1.z, s); s = fmaf(v1.w, v1.w, s);
            const float4 u0 = make_float4(v0.x * gain_s[r], v0.y * gain_s[r + 1], v0.z * gain_s[r + 2], v0.w * gain_s[r + 3]);
            const float4 u1 = make_float4(v1.x * gain_s[r + 4], v1.y * gain_s[r + 5], v1.z * gain_s[r + 6],
                                          v1.w * gain_s[r + 7]);
            bf16x8 hi, lo;
            split_hi_lo(u0, u1, hi, lo);
            const size_t i = split_index(m, row0 + r, MT);
            *reinterpret_cast<bf16x8 *>(a.us + i) = hi;
            *reinterpret_cast<bf16x8 *>(a.us + i + split_lo(MT)) = lo;
        }
        // the nc threads of a token are nc aligned consecutive lanes
        s += __shfl_xor(s, 1);
        s += __shfl_xor(s, 2);
        if (nc == 8) s += __shfl_xor(s, 4);
        if (e < total && (e & (nc - 1)) == 0) a.ssq_out[(size_t)(e / nc) * a.n_groups + group] = s;
    }
}

// SWIGLU on ntile consecutive tiles t0.. held in Y (tile p: gate rows at
// columns 32 p + [0,16), up rows at 32 p + 16 + [0,16)): h columns
// [16 t0, 16 (t0 + ntile)) of every token; in split layout 8 columns per
// thread (one 16-byte hi and one lo store).
__device__ void swiglu_epilogue(const GemmArgs &a, const float *Y, int ld, int t0, int ntile, const float *rinv)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    if (a.out_split) {
        const int MT = split_mt(a.Mpad, a.half), nc = 2 * ntile;
        for (int e = tid; e < split_rows(a.Mpad, a.half) * nc; e += nt) {
            const int m = e / nc, c = e - m * nc, p = c >> 1, r0 = 8 * (c & 1);
            const float *g = Y + m * ld + 32 * p + r0, *u = g + 16;
            float hv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) hv[i] = silu(g[i] * rinv[m]) * (u[i] * rinv[m]);
            bf16x8 hi, lo;
            split_hi_lo(make_float4(hv[0], hv[1], hv[2], hv[3]), make_float4(hv[4], hv[5], hv[6], hv[7]), hi, lo);
            const size_t i = split_index(m, 16 * t0 + 8 * c, MT);
            *reinterpret_cast<bf16x8 *>(a.out_split + i) = hi;
            *reinterpret_cast<bf16x8 *>(a.out_split + i + split_lo(MT)) = lo;
        }
    } else {
        for (int e = tid; e < a.Mpad * 16 * ntile; e += nt) {
            const int m = e / (16 * ntile), c = e - m * 16 * ntile, p = c >> 4, r = c & 15;
            const float hv = silu(Y[m * ld + 32 * p + r] * rinv[m]) * (Y[m * ld + 32 * p + 16 + r] * rinv[m]);
            a.out[(size_t)m * a.N + 16 * t0 + c] = hv;
        }
    }
}

// QKV on the 32-row tile t held in Y[m * ld + 0..32): rotary embedding of q
// and k at each token's position, q to the query buffer, k and v (rounded to
// the cache type) to cache slots P + m.
template <typename KV>
__device__ void qkv_epilogue(const GemmArgs &a, const float *Y, int ld, int t, const float *rinv)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    {
        const int per_seg = a.N / DV_GEMM_TILE;
        const int seg = t / per_seg, tt = t - seg * per_seg;
        const int per_head = a.hd / DV_GEMM_TILE;
        const int h = tt / per_head, j0 = (tt - h * per_head) * 16;
        const int half = a.hd / 2;
        for (int e = tid; e < a.M * 16; e += nt) {
            const int m = e / 16, r = e % 16;
            const int j = j0 + r;
            float y1 = Y[m * ld + r] * rinv[m], y2 = Y[m * ld + 16 + r] * rinv[m];
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
            } else {                // V: [H][cap/32][hd][32]
                KV *c = reinterpret_cast<KV *>(a.vc) + (size_t)h * a.hd * a.cap;
                Elem<KV>::store(c, v_index(j, a.P + m, a.hd), y1);
                Elem<KV>::store(c, v_index(j + half, a.P + m, a.hd), y2);
            }
        }
    }
}

// LOGITS: logits of rows [row0, row0 + nrows) and their per-token
// (max, argmax), lowest row on ties.
__device__ void logits_epilogue(const GemmArgs &a, const float *Y, int ld, int row0, int nrows, int group,
                                const float *rinv)
{
    const int tid = threadIdx.x, nt = blockDim.x;
    if (a.out) {
        for (int e = tid; e < a.M * nrows; e += nt) {
            const int m = e / nrows, r = e - m * nrows;
            a.out[(size_t)m * a.N + row0 + r] = Y[m * ld + r] * rinv[m];
        }
    }
    // 4 threads per token scan interleaved rows; combined by shuffles
    // (larger value, then lower row)
    if (tid < 4 * a.Mpad) {
        const int m = tid >> 2, c = tid & 3;
        const float ri = rinv[m];
        float best = -INFINITY;
        int bi = nrows;
        for (int r = c; r < nrows; r += 4) {
            const float v = Y[m * ld + r] * ri;
            if (v > best) { best = v; bi = r; }
        }
#pragma unroll
        for (int off = 1; off < 4; off <<= 1) {
            const float v2 = __shfl_xor(best, off);
            const int i2 = __shfl_xor(bi, off);
            if (v2 > best || (v2 == best && i2 < bi)) { best = v2; bi = i2; }
        }
        if (c == 0 && m < a.M) {
            a.arg_val[(size_t)m * a.n_groups + group] = best;
            a.arg_idx[(size_t)m * a.n_groups + group] = row0 + bi;
        }
    }
}

// PLAIN: rows [row0, row0 + nrows) of every token, 4 consecutive rows per
// thread.
__device__ void plain_epilogue(const GemmArgs &a, const float *Y, int ld, int row0, int nrows)
{
    const int nc = nrows >> 2;
    for (int e = threadIdx.x; e < a.M * nc; e += blockDim.x) {
        const int m = e / nc, r = 4 * (e - m * nc);
        const float *y = Y + m * ld + r;
        *reinterpret_cast<float4 *>(a.out + (size_t)m * a.N + row0 + r) = make_float4(y[0], y[1], y[2], y[3]);
    }
}

// ---------------------------------------------------------------------------
// MFMA projection for bf16 weights (block layout) and split-layout
// activations.
//
// v_mfma_f32_16x16x32_bf16: A = 16 weight rows x 32 k, B = 32 k x 16 tokens.
// Lane l supplies A[l%16][8(l/16)..+8] (16 contiguous bytes of one weight
// row) and B[8(l/16)..+8][l%16] for the bf16 hi and lo parts of the
// activations (two MFMAs per pair, so every product keeps ~16 mantissa bits
// of the fp32 activation).  D: lane l holds rows 4(l/16)..+4 of token l%16.
//
// Work unit = (row group g of RB blocks, K split ks); the NW waves take the
// unit's k-steps in turn (s = sb + wave, sb + wave + NW, ...), so a
// workgroup reads one RB KB stretch of each k-major slab; each wave keeps U
// k-steps of loads in flight (a new step is requested as soon as one is
// consumed).  The wave partials are summed in LDS in wave order.  A split
// unit stores its partial with device-coherent stores; the last unit of a
// row group to arrive (counted with a device-scope atomic, nobody waits) sums
// the ks partials in split order and runs the epilogue, so every sum has a
// fixed order and no workgroup ever waits for another.
//
// Loads: weights are read once per step (non-temporal hint), activations
// (MT KB hi + MT KB lo per k-step) are shared by every workgroup and stay in
// the caches.
//
// MT = 0: activations in the half split layout (at most 8 tokens): one 1 KB
// block per k-step carries hi in B columns 0-7 and lo in columns 8-15, so
// each weight block takes one MFMA and half the activation bytes; column n
// and column n + 8 are summed (a lane shuffle) once the unit's sums are
// complete, leaving columns 8-15 zero.

// Split-K partial slots hold this bit pattern (a NaN no arithmetic produces
// from finite inputs) while empty.  A folder reloads a chunk that still holds
// it: the arrival counter is bumped without waiting for the partial's stores,
// which are then still on their way; all empty chunks of a round are reloaded
// together.  The reload count is bounded so that a partial that really holds
// the pattern (NaN inputs) cannot stall the kernel.
#define DV_EMPTY_BITS 0xffffffffu
#define DV_EMPTY_SLOT ((u32x4){DV_EMPTY_BITS, DV_EMPTY_BITS, DV_EMPTY_BITS, DV_EMPTY_BITS})
#define DV_POLL_MAX 100000

__device__ __forceinline__ bool slot_empty(const u32x4 &r)
{
    return r[0] == DV_EMPTY_BITS || r[1] == DV_EMPTY_BITS || r[2] == DV_EMPTY_BITS || r[3] == DV_EMPTY_BITS;
}

#ifndef DV_WEIGHT_NT
#define DV_WEIGHT_NT 1
#endif
__device__ __forceinline__ u32x4 load_weights(const u32x4 *p)
{
    if (DV_WEIGHT_NT) return __builtin_nontemporal_load(p);
    return *p;
}

__global__ __launch_bounds__(64) void k_pack_blocks(GemmArgs a, int epi, uint16_t *dst)
{
    // grid: (row groups x rb blocks, k-step chunks)
    const int gb = blockIdx.x, lane = threadIdx.x;
    const int rb = a.rb, G = a.n_groups, S = a.K / 32;
    const int g = gb / rb, b = gb - g * rb;
    const RowMap rm = row_map(a, epi, gb >> 1);
    const int h = gb & 1;
    const uint16_t *src = reinterpret_cast<const uint16_t *>(rm.ptr[h]) +
                          (size_t)(rm.row0[h] + (lane & 15)) * a.K + (lane >> 4) * 8;
    for (int s = blockIdx.y; s < S; s += gridDim.y) {
        const uint4 v = *reinterpret_cast<const uint4 *>(src + 32 * s);
        *reinterpret_cast<uint4 *>(dst + (((size_t)s * G + g) * rb + b) * 512 + lane * 8) = v;
    }
}

// int8 weights: lane l of block (pair p, g, b) takes 8 bytes of k-step 2p and
// 8 bytes of k-step 2p + 1 of its row, so one 16-byte load feeds two MFMA
// k-steps.
__global__ __launch_bounds__(64) void k_pack_blocks_i8(GemmArgs a, int epi, uint8_t *dst)
{
    const int gb = blockIdx.x, lane = threadIdx.x;
    const int rb = a.rb, G = a.n_groups, S2 = a.K / 64;
    const int g = gb / rb, b = gb - g * rb;
    const RowMap rm = row_map(a, epi, gb >> 1);
    const int h = gb & 1;
    const int8_t *src = reinterpret_cast<const int8_t *>(rm.ptr[h]) + (size_t)(rm.row0[h] + (lane & 15)) * a.K +
                        (lane >> 4) * 8;
    for (int p = blockIdx.y; p < S2; p += gridDim.y) {
        const uint2 lo = *reinterpret_cast<const uint2 *>(src + 64 * p);
        const uint2 hi = *reinterpret_cast<const uint2 *>(src + 64 * p + 32);
        *reinterpret_cast<uint4 *>(dst + (((size_t)p * G + g) * rb + b) * 1024 + lane * 16) =
            make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
}

// Row scales in packed row order: block gb, row r -> dst[16 gb + r].
__global__ __launch_bounds__(16) void k_pack_scales(GemmArgs a, int epi, float *dst)
{
    const int gb = blockIdx.x, r = threadIdx.x;
    const RowMap rm = row_map(a, epi, gb >> 1);
    const int h = gb & 1;
    const float *sc = rm.mat[h] == 0 ? a.s0 : (rm.mat[h] == 1 ? a.s1 : a.s2);
    dst[gb * 16 + r] = sc[rm.row0[h] + r];
}

// Four int8 values -> four bf16 (exact: |q| <= 128 needs 8 significant bits),
// two per dword, low byte first.
__device__ __forceinline__ uint2 i8x4_to_bf16(uint32_t d)
{
    const uint32_t f0 = __float_as_uint((float)(int8_t)(d & 0xff));
    const uint32_t f1 = __float_as_uint((float)(int8_t)((d >> 8) & 0xff));
    const uint32_t f2 = __float_as_uint((float)(int8_t)((d >> 16) & 0xff));
    const uint32_t f3 = __float_as_uint((float)(int8_t)(d >> 24));
    return make_uint2(__builtin_amdgcn_perm(f1, f0, 0x07060302u), __builtin_amdgcn_perm(f3, f2, 0x07060302u));
}

template <int MT_, int EPI, typename KV, int NW, int U, int RB, bool Q8 = false>
__global__ __launch_bounds__(64 * NW) void k_proj(GemmArgs a)
{
    constexpr bool HALF = MT_ == 0;
    constexpr int MT = HALF ? 1 : MT_;  // token tiles of the MFMA outputs
    constexpr int ROWS = RB * 16, LD = ROWS + 1, NE = RB * MT * 64;
    static_assert(64 * NW >= 4 * 16 * MT, "input_rinv needs 4 threads per token");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tid = threadIdx.x;
    // a step is one k-step of 32 (bf16 weights) or a pair of them (int8);
    // XP activation blocks per step and token tile (PP parts per k-step)
    constexpr int PP = HALF ? 1 : 2, XP = (Q8 ? 2 : 1) * PP;
    const int S = a.K / (Q8 ? 64 : 32), G = a.n_groups, KS = a.ks;
    __shared__ f32x4 red[NW][NE / 64][64];
    __shared__ float Y[16 * MT * LD];
    __shared__ float rinv[DV_TREE_MAX];
    __shared__ int last_s;
    // RESID: the unit's rows of x (into Y) and their gains, staged while the
    // weights stream
    __shared__ float stage_s[EPI == EPI_RESID ? ROWS : 1];
    const u32x4 *Wb = reinterpret_cast<const u32x4 *>(a.packed);
    const u32x4 *Xb = reinterpret_cast<const u32x4 *>(a.xs);
    bool have_rinv = false;
    // Small epilogue operands (the input's norm partials, RESID: the unit's
    // rows of x and their gains, QKV: the rotary factors) are loaded into
    // registers before the unit's weight stream starts and consumed after it:
    // loads return in order, so they are back before the first weights and no
    // wait for them empties the stream.
    constexpr bool NEED_RINV = EPI != EPI_RESID && EPI != EPI_PLAIN;
    constexpr int NJP = MT >= 2 ? 8 : 24;                            // norm partials per thread
    constexpr int SXN = (16 * MT * ROWS + 64 * NW - 1) / (64 * NW);  // RESID: x values per thread
    // QKV and gate/up compute the input's 1/rms right after requesting their
    // first weight steps, so every wave waits for those steps before
    // streaming on; measured faster than preloading the partials (13B: QKV
    // 28.0 -> 26.9 us, gate/up 44.5 -> 43.6 us), while lm_head is faster
    // with the preload (51.4 against 53.2 us)
    constexpr bool RINV_FIRST = EPI == EPI_QKV || EPI == EPI_SWIGLU;
    static_assert(ROWS <= 64 * NW, "one gain per thread");

    for (int unit = blockIdx.x; unit < a.n_units; unit += gridDim.x) {
        const int g = unit / KS, ks = unit - g * KS;
        const int sb = (ks * S) / KS, se = ((ks + 1) * S) / KS;
        const int s0 = sb + wave;
        const int n = s0 < se ? (se - s0 + NW - 1) / NW : 0;
        auto wp = [&](int i, int b) -> const u32x4 * {
            return Wb + (((size_t)(s0 + NW * i) * G + g) * RB + b) * 64 + lane;
        };
        // activation block of step i, half hf (int8: k-step 2 step + hf), part q
        auto xp = [&](int i, int hf, int mt, int q) -> const u32x4 * {
            const size_t k32 = Q8 ? 2 * (size_t)(s0 + NW * i) + hf : (size_t)(s0 + NW * i);
            return Xb + ((k32 * MT + mt) * PP + q) * 64 + lane;
        };
        f32x4 acc[RB][MT];
#pragma unroll
        for (int b = 0; b < RB; ++b)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[b][mt] = (f32x4){0.f, 0.f, 0.f, 0.f};
        f32x4 rs[Q8 ? RB : 1];  // int8: this lane's four row scales per block
        float sx[EPI == EPI_RESID ? SXN : 1], sgain = 0.f;
        float sv[NEED_RINV ? NJP : 1];
        const bool load_rinv = NEED_RINV && !have_rinv;
        if constexpr (EPI == EPI_RESID) {
#pragma unroll
            for (int c = 0; c < SXN; ++c) {
                const int e = tid + 64 * NW * c, m = e / ROWS, r = e - m * ROWS;
                sx[c] = (e < 16 * MT * ROWS && m < a.M) ? a.resid[(size_t)m * a.N + g * ROWS + r] : 0.f;
            }
            if (tid < ROWS) sgain = Elem<uint16_t>::load(reinterpret_cast<const uint16_t *>(a.gain), g * ROWS + tid);
        }
        if constexpr (NEED_RINV && !RINV_FIRST) {
            if (load_rinv) rinv_load<NJP>(a, sv);
        }
        if (n > 0) {
            u32x4 wb[U][RB], xb[U][MT][XP];
            auto fetch = [&](int j, int i) {
#pragma unroll
                for (int b = 0; b < RB; ++b) wb[j][b] = load_weights(wp(i, b));
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int q = 0; q < XP; ++q) xb[j][mt][q] = *xp(i, q / PP, mt, q % PP);
            };
            auto mfma = [&](int j) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int hf = 0; hf < XP / PP; ++hf) {
                        const bf16x8 hi = __builtin_bit_cast(bf16x8, xb[j][mt][PP * hf]);
                        const bf16x8 lo = __builtin_bit_cast(bf16x8, xb[j][mt][PP * hf + PP - 1]);
#pragma unroll
                        for (int b = 0; b < RB; ++b) {
                            bf16x8 w;
                            if (Q8) {
                                const uint2 c0 = i8x4_to_bf16(wb[j][b][2 * hf]);
                                const uint2 c1 = i8x4_to_bf16(wb[j][b][2 * hf + 1]);
                                w = __builtin_bit_cast(bf16x8, (u32x4){c0.x, c0.y, c1.x, c1.y});
                            } else {
                                w = __builtin_bit_cast(bf16x8, wb[j][b]);
                            }
                            acc[b][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, hi, acc[b][mt], 0, 0, 0);
                            if (!HALF)
                                acc[b][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, lo, acc[b][mt], 0, 0, 0);
                        }
                    }
                }
            };
            // prologue: U steps in flight (indices past the end re-read the
            // last step and are dropped)
#pragma unroll
            for (int j = 0; j < U; ++j) fetch(j, min(j, n - 1));
            if (Q8) {
#pragma unroll
                for (int b = 0; b < RB; ++b)
                    rs[b] = *reinterpret_cast<const f32x4 *>(a.scale + (g * RB + b) * 16 + 4 * (lane >> 4));
            }
            if constexpr (RINV_FIRST) {
                // the first unit's weight steps are in flight
                if (!have_rinv) {
                    input_rinv(a, rinv);
                    have_rinv = true;
                }
            }
            int i = 0;
            for (; i + U < n; i += U) {
#pragma unroll
                for (int j = 0; j < U; ++j) {
                    mfma(j);
                    fetch(j, min(i + j + U, n - 1));
                    // keep step j's loads ahead of step j + 1's MFMAs: the
                    // scheduler would otherwise move every load of the round
                    // behind the last MFMA, emptying the pipeline each round
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
#pragma unroll
            for (int j = 0; j < U; ++j)
                if (i + j < n) mfma(j);
            if (Q8) {
                // W = scale[row] q: scale this wave's sums row by row
#pragma unroll
                for (int b = 0; b < RB; ++b)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) acc[b][mt] *= rs[b];
            }
        }
        // the epilogue operands loaded before the stream, into LDS
        if constexpr (EPI == EPI_RESID) {
#pragma unroll
            for (int c = 0; c < SXN; ++c) {
                const int e = tid + 64 * NW * c, m = e / ROWS, r = e - m * ROWS;
                if (e < 16 * MT * ROWS) Y[m * LD + r] = sx[c];
            }
            if (tid < ROWS) stage_s[tid] = sgain;
        }
        if constexpr (NEED_RINV && !RINV_FIRST) {
            if (load_rinv) {
                rinv_finish<NJP>(a, sv, rinv);
                have_rinv = true;
            }
        }
        if constexpr (RINV_FIRST) {
            if (!have_rinv) {  // a unit without k-steps for this workgroup's waves
                input_rinv(a, rinv);
                have_rinv = true;
            }
        }

        // wave partials -> unit sums (fixed wave order)
#pragma unroll
        for (int b = 0; b < RB; ++b)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) red[wave][b * MT + mt][lane] = acc[b][mt];
        __syncthreads();
        f32x4 v[(NE + 64 * NW - 1) / (64 * NW)];
#pragma unroll
        for (int c = 0; c < (NE + 64 * NW - 1) / (64 * NW); ++c) {
            const int e = tid + 64 * NW * c;
            v[c] = (f32x4){0.f, 0.f, 0.f, 0.f};
            if (e < NE) {
                v[c] = red[0][e >> 6][e & 63];
#pragma unroll
                for (int w = 1; w < NW; ++w) v[c] += red[w][e >> 6][e & 63];
            }
        }
        bool mine = true;
        if (KS > 1) {
            // Count this split's arrival first; the last split to arrive
            // folds, the others publish their partials (16-byte stores
            // written through to the device-coherent level, cache policy
            // sc1).  The folder takes its own partial from registers and
            // loads the others, reloading a chunk while it still holds the
            // empty-slot pattern (every slot holds it between launches: the
            // folder puts it back after reading), so no split ever waits for
            // its own stores.
            const __amdgpu_buffer_rsrc_t pr =
                __builtin_amdgcn_make_buffer_rsrc(a.part, (short)0, 0x7fffffff, 0x00020000);
            if (tid == 0) {
                const uint32_t old = __hip_atomic_fetch_add(a.cnt + g, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                last_s = old == (uint32_t)(KS - 1);
            }
            __syncthreads();
            mine = last_s != 0;
#pragma unroll
            for (int c = 0; c < (NE + 64 * NW - 1) / (64 * NW); ++c) {
                const int e = tid + 64 * NW * c;
                if (e >= NE) continue;
                if (!mine) {
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v[c]), pr,
                                                           (uint32_t)(((size_t)unit * NE + e) * 16), 0, 16);
                    continue;
                }
                // fold in split order, loads of 4 splits in flight together
                f32x4 sum = (f32x4){0.f, 0.f, 0.f, 0.f};
                for (int k0 = 0; k0 < KS; k0 += 4) {
                    u32x4 raw[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int k = k0 + j;
                        if (k < KS && k != ks)
                            raw[j] = __builtin_amdgcn_raw_buffer_load_b128(
                                pr, (uint32_t)(((size_t)(g * KS + k) * NE + e) * 16), 0, 16);
                    }
                    // reload every chunk still empty, all together, until none is
                    for (int it = 0; it < DV_POLL_MAX; ++it) {
                        bool any = false;
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            any |= k0 + j < KS && k0 + j != ks && slot_empty(raw[j]);
                        if (!any) break;
                        __builtin_amdgcn_s_sleep(1);
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int k = k0 + j;
                            if (k < KS && k != ks && slot_empty(raw[j]))
                                raw[j] = __builtin_amdgcn_raw_buffer_load_b128(
                                    pr, (uint32_t)(((size_t)(g * KS + k) * NE + e) * 16), 0, 16);
                        }
                    }
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int k = k0 + j;
                        if (k >= KS) break;
                        if (k == ks) {
                            sum += v[c];
                        } else {
                            sum += __builtin_bit_cast(f32x4, raw[j]);
                            __builtin_amdgcn_raw_buffer_store_b128(
                                DV_EMPTY_SLOT, pr, (uint32_t)(((size_t)(g * KS + k) * NE + e) * 16), 0, 16);
                        }
                    }
                }
                v[c] = sum;
            }
            if (mine && tid == 0) __hip_atomic_store(a.cnt + g, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (mine) {
            if (HALF) {
                // token n = hi column n + lo column n + 8; columns 8-15 -> 0
                // (every lane of a wave holds the same e >> 6)
#pragma unroll
                for (int c = 0; c < (NE + 64 * NW - 1) / (64 * NW); ++c)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float o = __shfl_xor(v[c][j], 8);
                        v[c][j] = (lane & 8) ? 0.f : v[c][j] + o;
                    }
            }
            // D layout -> Y[token][row]
#pragma unroll
            for (int c = 0; c < (NE + 64 * NW - 1) / (64 * NW); ++c) {
                const int e = tid + 64 * NW * c;
                if (e < NE) {
                    const int l = e & 63, bm = e >> 6, b = bm / MT, mt = bm - b * MT;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        float &y = Y[(mt * 16 + (l & 15)) * LD + b * 16 + 4 * (l >> 4) + j];
                        y = EPI == EPI_RESID ? y + v[c][j] : v[c][j];
                    }
                }
            }
            __syncthreads();
            if (EPI == EPI_RESID) {
                if (a.us) resid_epilogue_split(a, Y, LD, g * ROWS, ROWS, g, stage_s);
                else resid_epilogue<uint16_t>(a, Y, LD, g * ROWS, ROWS, g, true, stage_s);
            } else if (EPI == EPI_LOGITS) {
                logits_epilogue(a, Y, LD, g * ROWS, ROWS, g, rinv);
            } else if (EPI == EPI_PLAIN) {
                plain_epilogue(a, Y, LD, g * ROWS, ROWS);
            } else if (EPI == EPI_SWIGLU) {
                swiglu_epilogue(a, Y, LD, g * (RB / 2), RB / 2, rinv);
            } else {
#pragma unroll
                for (int p = 0; p < RB / 2; ++p) qkv_epilogue<KV>(a, Y + 32 * p, LD, g * (RB / 2) + p, rinv);
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// VALU GEMM (fp32 weights, or bf16 where K is not a multiple of 32).  One
// 32-row tile per unit, full K.  Thread (row r = tid/8, lane-in-row kl =
// tid%8) walks k = 8 kl + 64 i, 8 weights per load; 16 tokens per pass; the 8
// partial sums of a row are combined with butterfly shuffles.

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
    constexpr int LD = DV_GEMM_TILE + 1;
    const int r = threadIdx.x >> 3, kl = threadIdx.x & 7;
    const int K = a.K;
    __shared__ float Y[DV_TREE_MAX * LD];
    __shared__ float rinv[DV_TREE_MAX];
    if (EPI != EPI_RESID) {
        input_rinv(a, rinv);
        __syncthreads();
    }
    for (int t = blockIdx.x; t < a.n_tiles; t += gridDim.x) {
        const RowMap rm = row_map(a, EPI, t);
        const int hsel = r >> 4;
        const W *wrow = reinterpret_cast<const W *>(rm.ptr[hsel]) + (size_t)(rm.row0[hsel] + (r & 15)) * K;
        for (int m0 = 0; m0 < a.Mpad; m0 += 16) {
            float acc[16];
#pragma unroll
            for (int m = 0; m < 16; ++m) acc[m] = 0.f;
            for (int k = kl * 8; k < K; k += 64) {
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
                if (kl == 0) Y[(m0 + m) * LD + r] = v;
            }
        }
        __syncthreads();
        if (EPI == EPI_RESID) resid_epilogue<W>(a, Y, LD, t * DV_GEMM_TILE, DV_GEMM_TILE, t, false, nullptr);
        else if (EPI == EPI_LOGITS) logits_epilogue(a, Y, LD, t * DV_GEMM_TILE, DV_GEMM_TILE, t, rinv);
        else if (EPI == EPI_SWIGLU) swiglu_epilogue(a, Y, LD, t, 1, rinv);
        else qkv_epilogue<KV>(a, Y, LD, t, rinv);
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// First RMSNorm of the step: grid (Mpad rows, DV_NORM_SLICES column slices),
// rows in [M, Mpad) are written as 0.  x = embedding row of the token; u = x
// * gain; the slice's sum of squares.

template <typename W, int NV>
__global__ __launch_bounds__(DV_NORM_THREADS) void k_embed_norm(NormArgs a)
{
    constexpr int NT = DV_NORM_THREADS, SPAN = 4 * NT;
    const int m = blockIdx.x, sl = blockIdx.y, tid = threadIdx.x, d = a.d;
    const int c0 = sl * (d / DV_NORM_SLICES), c1 = c0 + d / DV_NORM_SLICES;
    float *urow = a.u + (size_t)m * d;
    float *xrow = a.x + (size_t)m * d;
    const int MT = split_mt(gridDim.x, a.half);  // grid.x = Mpad rows
    if (m >= a.M) {
        for (int i = c0 + 4 * tid; i < c1; i += SPAN) {
            const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
            if (a.us) {
                if (m < split_rows(gridDim.x, a.half)) store_split4(a.us, m, i, MT, z);
            } else {
                *reinterpret_cast<float4 *>(urow + i) = z;
            }
            *reinterpret_cast<float4 *>(xrow + i) = z;
        }
        if (tid == 0) a.ssq[m * DV_NORM_SLICES + sl] = 0.f;
        return;
    }
    // NV = ceil(slice / SPAN) float4 per thread; addresses are clamped, not
    // branched on: lanes past the slice end re-read its last float4 and drop it
    int idx[NV];
#pragma unroll
    for (int c = 0; c < NV; ++c) idx[c] = min(c0 + 4 * tid + SPAN * c, c1 - 4);
    float4 v[NV];
    if (a.x_in) {  // input rows given (the draft's fused inputs)
#pragma unroll
        for (int c = 0; c < NV; ++c) v[c] = *reinterpret_cast<const float4 *>(a.x_in + (size_t)m * d + idx[c]);
    } else {
        const W *e = reinterpret_cast<const W *>(a.embed) + (size_t)a.tokens[m] * d;
#pragma unroll
        for (int c = 0; c < NV; ++c)
            v[c] = make_float4(Elem<W>::load(e, idx[c]), Elem<W>::load(e, idx[c] + 1),
                               Elem<W>::load(e, idx[c] + 2), Elem<W>::load(e, idx[c] + 3));
    }
    const W *gp = reinterpret_cast<const W *>(a.gain);
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NV; ++c) {
        const int i = idx[c];
        if (c0 + 4 * tid + SPAN * c < c1) {
            *reinterpret_cast<float4 *>(xrow + i) = v[c];
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
// Cache layouts: K [H][cap][hd] (key-major), V [H][cap/32][hd][32] (32-slot
// tiles, dim-major within a tile; see v_index).
// Workgroup (split s, head h) covers keys [s*kps, (s+1)*kps) of the P + M
// cache slots; the tree's own keys/values were written to slots P.. by the
// QKV epilogue.  Key j is visible to node i iff j < P or bit (j-P) of
// anc(i).  Each split writes its unnormalised output with the running max
// and sum; the splits are combined by the last split of the head to finish
// (bf16 cache) or by k_attn_merge (fp32 cache); with one split the workgroup
// writes the normalised output itself.

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
// exponential is one exp2 (the running max handed to the merge stays in
// base-2 units).  Each wave keeps two tiles of K and V in
// registers (the next one loads while the current one is used); the
// prologue issues the query, ancestor-mask and first-tile loads together.

// DB: two register tiles per wave (next tile loads while the current one is
// used; for long key ranges); without DB every wave holds one tile, which
// leaves room for 8 waves when a split has at most one tile per wave.
// QT query tiles of 16 are held at once (M <= 16 QT): every loaded key tile
// serves all of them, each with its own running max, sum and output.
template <int HD, int NW, bool DB, int QT>
__global__ __launch_bounds__(64 * NW) void k_attn_mfma(AttnArgs a)
{
    constexpr int NC = HD / 32;  // QK k-steps over dims
    constexpr int ND = HD / 16;  // PV output dim tiles
    static_assert(64 * NW >= 2 * HD, "one thread per 8 query values");
    const int split = blockIdx.x, h = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n = lane & 15, g = lane >> 4;
    const int M = a.tm.M, P = a.tm.P, total = P + M;
    const int kbeg = split * a.keys_per_split;
    const int kend = min(total, kbeg + a.keys_per_split);
    const int ntile = (kend - kbeg + 31) / 32;
    const int D = a.H * HD;
    const float scale2 = 1.4426950408889634f / sqrtf((float)HD);
    const uint16_t *kc = reinterpret_cast<const uint16_t *>(a.kc) + (size_t)h * a.cap * HD;
    const uint16_t *vc = reinterpret_cast<const uint16_t *>(a.vc) + (size_t)h * HD * a.cap;
    // split partials (device-coherent 16-byte stores and loads)
    const __amdgpu_buffer_rsrc_t po = __builtin_amdgcn_make_buffer_rsrc(a.part_o, (short)0, 0x7fffffff, 0x00020000);

    __shared__ u32x4 sm_q[QT][NC * 2 * 64];  // per query tile: [k-step][hi/lo][lane] B operands
    __shared__ float sm_m[NW][16], sm_l[NW][16];
    __shared__ __align__(16) float sm_o[NW][16][HD + 4];

    struct Tile {
        u32x4 ka[NC], kb[NC], v[ND];
    };
    // keys and values are read once per step: non-temporal loads
    auto load = [&](int t, Tile &T) {
        const int k0 = kbeg + 32 * t;
        const int ka = min(k0 + 8 * (n >> 2) + (n & 3), kend - 1);
        const int kb = min(k0 + 8 * (n >> 2) + 4 + (n & 3), kend - 1);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            T.ka[c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(kc + (size_t)ka * HD + 32 * c + 8 * g));
            T.kb[c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(kc + (size_t)kb * HD + 32 * c + 8 * g));
        }
        // columns past the last cache slot of the tile stay inside the
        // allocation (capacity is a multiple of 32); they are masked below
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
            T.v[dt] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4 *>(vc + ((size_t)(k0 >> 5) * HD + dt * 16 + n) * 32 + 8 * g));
    };

    // queries of all tiles into LDS (hi + lo B operands) with the first key
    // tile's loads in flight
    Tile buf0;
    Tile buf1;  // used with DB only
    if (wave < ntile) load(wave, buf0);
    uint64_t anc[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int tok = 16 * qt + n;
        anc[qt] = tok < M ? a.tm.anc[tok] : 0ull;
        // thread e < 2*HD converts 8 dims (c, group qg) of query row qr
        const int e = threadIdx.x;
        const int qr = e / (2 * NC * 2) % 16, qc = (e >> 2) % NC, qg = e & 3;
        if (e < 2 * HD) {
            const int row = 16 * qt + qr;
            float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
            if (row < M) {
                const float *qp = a.q + (size_t)row * D + h * HD + qc * 32 + qg * 8;
                x0 = *reinterpret_cast<const float4 *>(qp);
                x1 = *reinterpret_cast<const float4 *>(qp + 4);
            }
            bf16x8 hh, ll;
            split_hi_lo(x0, x1, hh, ll);
            sm_q[qt][(qc * 2 + 0) * 64 + 16 * qg + qr] = __builtin_bit_cast(u32x4, hh);
            sm_q[qt][(qc * 2 + 1) * 64 + 16 * qg + qr] = __builtin_bit_cast(u32x4, ll);
        }
    }
    __syncthreads();

    float m_run[QT], l_run[QT];
    f32x4 o[QT][ND];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m_run[qt] = -INFINITY;
        l_run[qt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) o[qt][dt] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }

    auto process = [&](int t, Tile &cur) {
        const int k0 = kbeg + 32 * t;
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
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            if (16 * qt >= M) break;
            f32x4 sa = (f32x4){0.f, 0.f, 0.f, 0.f}, sb = sa;
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const bf16x8 ka8 = __builtin_bit_cast(bf16x8, cur.ka[c]);
                const bf16x8 kb8 = __builtin_bit_cast(bf16x8, cur.kb[c]);
                const bf16x8 qh = __builtin_bit_cast(bf16x8, sm_q[qt][(c * 2 + 0) * 64 + lane]);
                const bf16x8 ql = __builtin_bit_cast(bf16x8, sm_q[qt][(c * 2 + 1) * 64 + lane]);
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
                const bool tree_ok = sh < 0 || ((anc[qt] >> (sh & 63)) & 1ull);
                const bool vis = key < kend && tree_ok;
                const float sc = (i < 4 ? sa[i] : sb[i - 4]) * scale2;
                sv[i] = vis ? sc : -INFINITY;
                mt = fmaxf(mt, sv[i]);
            }
            mt = fmaxf(mt, __shfl_xor(mt, 16));
            mt = fmaxf(mt, __shfl_xor(mt, 32));
            const float mnew = fmaxf(m_run[qt], mt);
            const float alpha = m_run[qt] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[qt] - mnew);
            float ps = 0.f, pv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                pv[i] = sv[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sv[i] - mnew);
                ps += pv[i];
            }
            ps += __shfl_xor(ps, 16);
            ps += __shfl_xor(ps, 32);
            l_run[qt] = l_run[qt] * alpha + ps;
            m_run[qt] = mnew;
            // O rows held by this lane are tokens 4g + j of the tile
            float al[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) al[j] = __shfl(alpha, 4 * g + j);
            bf16x8 ph, pl;
            split_hi_lo(make_float4(pv[0], pv[1], pv[2], pv[3]), make_float4(pv[4], pv[5], pv[6], pv[7]), ph, pl);
#pragma unroll
            for (int dt = 0; dt < ND; ++dt) {
#pragma unroll
                for (int j = 0; j < 4; ++j) o[qt][dt][j] *= al[j];
                const bf16x8 v8 = __builtin_bit_cast(bf16x8, cur.v[dt]);
                o[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, v8, o[qt][dt], 0, 0, 0);
                o[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, v8, o[qt][dt], 0, 0, 0);
            }
        }
    };
    if (DB) {
        // two register buffers used in turn (no copies between them, so a
        // load in flight is never waited on before its tile is used)
        for (int t = wave; t < ntile; t += 2 * NW) {
            if (t + NW < ntile) load(t + NW, buf1);
            process(t, buf0);
            if (t + NW >= ntile) break;
            if (t + 2 * NW < ntile) load(t + 2 * NW, buf0);
            process(t + NW, buf1);
        }
    } else {
        for (int t = wave; t < ntile; t += NW) {
            if (t != wave) load(t, buf0);
            process(t, buf0);
        }
    }

    // combine the waves (fixed wave order), one query tile at a time
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        if (16 * qt >= M) break;
        if (g == 0) {
            sm_m[wave][n] = m_run[qt];
            sm_l[wave][n] = l_run[qt];
        }
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
#pragma unroll
            for (int j = 0; j < 4; ++j) sm_o[wave][4 * g + j][dt * 16 + n] = o[qt][dt][j];
        __syncthreads();
        // 4 consecutive dims of one node per thread
        for (int e4 = threadIdx.x; e4 < 16 * (HD / 4); e4 += 64 * NW) {
            const int i = e4 / (HD / 4), d0 = 4 * (e4 % (HD / 4));
            const int ti = 16 * qt + i;
            float mx = -INFINITY;
#pragma unroll
            for (int w = 0; w < NW; ++w) mx = fmaxf(mx, sm_m[w][i]);
            float l = 0.f;
            f32x4 ov = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int w = 0; w < NW; ++w) {
                const float mw = sm_m[w][i];
                const float wgt = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - mx);
                l = fmaf(wgt, sm_l[w][i], l);
                const f32x4 o4 = *reinterpret_cast<const f32x4 *>(&sm_o[w][i][d0]);
#pragma unroll
                for (int j = 0; j < 4; ++j) ov[j] = fmaf(wgt, o4[j], ov[j]);
            }
            if (a.n_split == 1) {
                if (ti < (a.out_split ? split_rows(a.tm.Mpad, a.tm.half) : a.tm.Mpad)) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float r = ti < M ? ov[j] / l : 0.f;
                        if (a.out_split)
                            store_split(a.out_split, ti, h * HD + d0 + j, split_mt(a.tm.Mpad, a.tm.half), r);
                        else a.out[(size_t)ti * D + h * HD + d0 + j] = r;
                    }
                }
            } else if (ti < M) {
                // published with device-coherent stores for the merging workgroup
                const size_t pb = ((size_t)h * a.n_split + split) * DV_TREE_MAX + ti;
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, ov), po, (uint32_t)((pb * HD + d0) * 4),
                                                       0, 16);
                if (d0 == 0) {
                    __hip_atomic_store(a.part_m + pb, mx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(a.part_l + pb, l, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
        __syncthreads();
    }
    if (a.n_split == 1) return;

    // The last split of this head to finish (device-scope counter; nobody
    // waits) merges the splits of every node in split order: a softmax-
    // weighted sum with a running maximum (base-2 units), then the output in
    // split layout, 8 dims of one node per thread.
    // (the partials were published without waiting for the stores: the
    // merging split reloads any value that still holds the empty-slot
    // pattern, and empties every slot it read for the next launch)
    __shared__ int last_s;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t old = __hip_atomic_fetch_add(a.cnt + h, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last_s = old == (uint32_t)(a.n_split - 1);
    }
    __syncthreads();
    if (!last_s) return;
    const int MT = split_mt(a.tm.Mpad, a.tm.half);
    const int rows = a.out_split ? split_rows(a.tm.Mpad, a.tm.half) : a.tm.Mpad;
    constexpr int CH = 8;  // splits whose loads are in flight together
    for (int e2 = threadIdx.x; e2 < rows * (HD / 8); e2 += 64 * NW) {
        const int i = e2 / (HD / 8), d0 = 8 * (e2 % (HD / 8));
        float ov[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        float run_m = -INFINITY, l = 0.f;
        if (i < M) {
            for (int s0 = 0; s0 < a.n_split; s0 += CH) {
                float ms[CH], ls[CH];
                f32x4 oa[CH], ob[CH];
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    const size_t pb = ((size_t)h * a.n_split + min(s0 + c, a.n_split - 1)) * DV_TREE_MAX + i;
                    ms[c] = __hip_atomic_load(a.part_m + pb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    ls[c] = __hip_atomic_load(a.part_l + pb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    const uint32_t off = (uint32_t)((pb * HD + d0) * 4);
                    oa[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(po, off, 0, 16));
                    ob[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(po, off + 16, 0, 16));
                }
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    if (s0 + c >= a.n_split || ms[c] == -INFINITY) continue;
                    const float mx = fmaxf(run_m, ms[c]);
                    const float sc = run_m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(run_m - mx);
                    const float w = __builtin_amdgcn_exp2f(ms[c] - mx);
                    l = fmaf(w, ls[c], l * sc);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        ov[j] = fmaf(w, oa[c][j], ov[j] * sc);
                        ov[4 + j] = fmaf(w, ob[c][j], ov[4 + j] * sc);
                    }
                    run_m = mx;
                }
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) ov[j] /= l;
        }
        if (a.out_split) {
            bf16x8 hi, lo;
            split_hi_lo(make_float4(ov[0], ov[1], ov[2], ov[3]), make_float4(ov[4], ov[5], ov[6], ov[7]), hi, lo);
            const size_t si = split_index(i, h * HD + d0, MT);
            *reinterpret_cast<bf16x8 *>(a.out_split + si) = hi;
            *reinterpret_cast<bf16x8 *>(a.out_split + si + split_lo(MT)) = lo;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) a.out[(size_t)i * D + h * HD + d0 + j] = ov[j];
        }
    }
    if (threadIdx.x == 0) __hip_atomic_store(a.cnt + h, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// fp32 cache (VALU).  K/V tiles of 32 keys sit in LDS as fp32; 16 queries
// at a time; an online softmax keeps (max, sum, o) per query.

template <int HD>
__global__ __launch_bounds__(256) void k_attn_f32(AttnArgs a)
{
    constexpr int DPT = HD / 16;  // output dims per thread
    const int split = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const int M = a.tm.M, P = a.tm.P, total = P + M;
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
                vt[jv][dv] = jv < nk ? vc[v_index(dv, t0 + jv, HD)] : 0.f;
            }
            __syncthreads();
            for (int e = tid; e < 16 * DV_ATTN_TILE; e += 256) {
                const int i = e / DV_ATTN_TILE, j = e % DV_ATTN_TILE;
                const int key = t0 + j;
                bool vis = i < nq && j < nk;
                if (vis && key >= P) vis = (a.tm.anc[q0 + i] >> (key - P)) & 1ull;
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
            if (q0 + qi < (a.out_split ? split_rows(a.tm.Mpad, a.tm.half) : a.tm.Mpad)) {
#pragma unroll
                for (int c = 0; c < DPT; ++c) {
                    const float r = qi < nq ? o[c] / lrun[qi] : 0.f;
                    if (a.out_split)
                        store_split(a.out_split, q0 + qi, h * HD + dd + c, split_mt(a.tm.Mpad, a.tm.half), r);
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
    const int M = a.tm.M, MT = split_mt(gridDim.x, a.tm.half);
    if (i >= M) {
        if (a.out_split) {
            if (i < split_rows(gridDim.x, a.tm.half)) store_split(a.out_split, i, h * HD + d, MT, 0.f);
        }
        else {
            a.out[(size_t)i * a.H * HD + h * HD + d] = 0.f;
        }
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
    const int M = a.M, tid = threadIdx.x;
    // tpt threads per node (64, 32 or 16) scan the partials with stride tpt
    // (neighbouring lanes read neighbouring entries), 16 loads in flight
    // (clamped indices only repeat a real entry)
    const int tpt = a.Mpad <= 16 ? 64 : (a.Mpad <= 32 ? 32 : 16);
    const int m = tid / tpt, sub = tid % tpt;
    if (m < M) {
        const float *val = a.arg_val + (size_t)m * a.n_parts;
        const int32_t *idx = a.arg_idx + (size_t)m * a.n_parts;
        float best = -INFINITY;
        int bi = 0x7fffffff;
        for (int t = sub; t < a.n_parts; t += 16 * tpt) {
            float v[16];
            int ix[16];
#pragma unroll
            for (int c = 0; c < 16; ++c) {
                const int tt = min(t + c * tpt, a.n_parts - 1);
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
        par_s[tid] = a.parents[tid];
        tok_s[tid] = a.tokens[tid];
        dep_s[tid] = a.depth[tid];
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
// Sampled acceptance (temperature > 0), one workgroup of 1024 threads walking
// the tree.  Thread i owns the vocabulary chunk [i ch, i ch + ch), ch a
// multiple of 4; every total is the chunk summed in id order followed by a
// fixed butterfly / wave-order combine, so a run is deterministic.  The
// current distribution is kept unnormalised (P and its total S) in one of two
// workspace rows, so a rejected child forms its residual without a division:
// child token t is accepted iff u q(t) S < P(t); the residual is
// R = max(P - q S, 0), adopted only when its total is positive.  The bonus is
// the first id whose running mass exceeds u_bonus times the total.

constexpr int SAMPLE_THREADS = 1024;

// Block-wide reduction of one value per thread (OP: 0 sum, 1 max, 2 min),
// identical in every thread: a butterfly within each wave, then the wave
// results in wave order.
template <int OP, typename T>
__device__ __forceinline__ T red_op(T a, T b)
{
    return OP == 0 ? a + b : (OP == 1 ? (a > b ? a : b) : (a < b ? a : b));
}

template <int OP, typename T>
__device__ __forceinline__ T block_reduce(T v, T *red)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = red_op<OP>(v, __shfl_xor(v, off));
    __syncthreads();  // red[] is free again
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    T r = red[0];
#pragma unroll
    for (int w = 1; w < SAMPLE_THREADS / 64; ++w) r = red_op<OP>(r, red[w]);
    return r;
}

// Up to SAMPLE_BATCH float4 of a thread's chunk, all loads issued before any
// is used (entries past v1 read as `fill`).
constexpr int SAMPLE_BATCH = 8;

__device__ __forceinline__ void load_batch(const float *base, int v, int v1, float fill,
                                           float4 (&t)[SAMPLE_BATCH])
{
#pragma unroll
    for (int j = 0; j < SAMPLE_BATCH; ++j) {
        const int vv = v + 4 * j;
        t[j] = vv < v1 ? reinterpret_cast<const float4 *>(base)[vv >> 2] : make_float4(fill, fill, fill, fill);
    }
}

__global__ __launch_bounds__(SAMPLE_THREADS) void k_accept_sampled(SampleArgs a)
{
    __shared__ float red[SAMPLE_THREADS / 64];
    __shared__ int ired[SAMPLE_THREADS / 64];
    __shared__ float scan_w[SAMPLE_THREADS / 64];
    __shared__ int32_t par_s[DV_TREE_MAX], tok_s[DV_TREE_MAX], path_s[DV_TREE_MAX];
    __shared__ float ua_s[DV_TREE_MAX], ub_s[DV_TREE_MAX];
    const int tid = threadIdx.x, V = a.V, M = a.M;
    if (tid < M) {
        par_s[tid] = a.parents[tid];
        tok_s[tid] = a.tokens[tid];
        ua_s[tid] = a.u_accept[tid];
        ub_s[tid] = a.u_bonus[tid];
    }
    if (tid == 0) path_s[0] = 0;
    const int ch = ((V + 4 * SAMPLE_THREADS - 1) / (4 * SAMPLE_THREADS)) * 4;
    const int v0 = min(tid * ch, V), v1 = min(v0 + ch, V);
    const float k2 = a.inv_t * 1.4426950408889634f;  // exp(x / T) = 2^(x log2(e) / T)
    float *P = a.p, *Pn = a.p + V;
    float S = 0.f;
    int cur = 0, n = 1;

    // P <- exp((z - max z) / T) of the logits row at node `node`, S <- its
    // total.  The first batch of the chunk (the whole chunk up to a
    // 32768-id vocabulary) stays in registers between the two passes.
    auto load_dist = [&](int node) {
        const float *z = a.logits + (size_t)node * V;
        float4 t0[SAMPLE_BATCH], t[SAMPLE_BATCH];
        load_batch(z, v0, v1, -INFINITY, t0);
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < SAMPLE_BATCH; ++j) mx = fmaxf(mx, fmaxf(fmaxf(t0[j].x, t0[j].y), fmaxf(t0[j].z, t0[j].w)));
        for (int v = v0 + 4 * SAMPLE_BATCH; v < v1; v += 4 * SAMPLE_BATCH) {
            load_batch(z, v, v1, -INFINITY, t);
#pragma unroll
            for (int j = 0; j < SAMPLE_BATCH; ++j) mx = fmaxf(mx, fmaxf(fmaxf(t[j].x, t[j].y), fmaxf(t[j].z, t[j].w)));
        }
        mx = block_reduce<1>(mx, red);
        float sum = 0.f;
        for (int v = v0; v < v1; v += 4 * SAMPLE_BATCH) {
            if (v != v0) load_batch(z, v, v1, -INFINITY, t);
#pragma unroll
            for (int j = 0; j < SAMPLE_BATCH; ++j) {
                const float4 x = v == v0 ? t0[j] : t[j];
                if (v + 4 * j < v1) {
                    float4 e;
                    e.x = exp2f((x.x - mx) * k2);
                    e.y = exp2f((x.y - mx) * k2);
                    e.z = exp2f((x.z - mx) * k2);
                    e.w = exp2f((x.w - mx) * k2);
                    reinterpret_cast<float4 *>(P)[(v >> 2) + j] = e;
                    sum += e.x + e.y + e.z + e.w;
                }
            }
        }
        S = block_reduce<0>(sum, red);  // its barriers also publish P
    };

    load_dist(0);
    int c = 1;
    while (true) {
        while (c < M && par_s[c] != cur) ++c;
        if (c >= M) break;  // no child of cur left: stop here
        const float *qu = a.q + (size_t)cur * V;
        const int t = tok_s[c];
        if (ua_s[c] * qu[t] * S < P[t]) {
            if (tid == 0) path_s[n] = c;
            ++n;
            cur = c;
            load_dist(cur);
            c = cur + 1;
            continue;
        }
        // rejected: residual of the current distribution
        float sum = 0.f;
        for (int v = v0; v < v1; v += 4 * SAMPLE_BATCH) {
            float4 pv[SAMPLE_BATCH], qv[SAMPLE_BATCH];
            load_batch(P, v, v1, 0.f, pv);
            load_batch(qu, v, v1, 0.f, qv);
#pragma unroll
            for (int j = 0; j < SAMPLE_BATCH; ++j) {
                if (v + 4 * j < v1) {
                    float4 r;
                    r.x = fmaxf(pv[j].x - qv[j].x * S, 0.f);
                    r.y = fmaxf(pv[j].y - qv[j].y * S, 0.f);
                    r.z = fmaxf(pv[j].z - qv[j].z * S, 0.f);
                    r.w = fmaxf(pv[j].w - qv[j].w * S, 0.f);
                    reinterpret_cast<float4 *>(Pn)[(v >> 2) + j] = r;
                    sum += r.x + r.y + r.z + r.w;
                }
            }
        }
        const float S2 = block_reduce<0>(sum, red);
        if (S2 > 0.f) {
            float *tmp = P;
            P = Pn;
            Pn = tmp;
            S = S2;
        }
        ++c;
    }

    // bonus: inclusive scan of the chunk totals in thread order, then each
    // thread walks its own chunk from its exclusive prefix
    float own = 0.f;
    for (int v = v0; v < v1; v += 4 * SAMPLE_BATCH) {
        float4 pv[SAMPLE_BATCH];
        load_batch(P, v, v1, 0.f, pv);
#pragma unroll
        for (int j = 0; j < SAMPLE_BATCH; ++j) own += pv[j].x + pv[j].y + pv[j].z + pv[j].w;
    }
    const int lane = tid & 63, wv = tid >> 6;
    float inc = own;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const float o = __shfl_up(inc, off);
        if (lane >= off) inc += o;
    }
    if (lane == 63) scan_w[wv] = inc;
    __syncthreads();
    float wbase = 0.f, total = 0.f;
    for (int w = 0; w < SAMPLE_THREADS / 64; ++w) {
        if (w < wv) wbase += scan_w[w];
        total += scan_w[w];
    }
    const float target = ub_s[cur] * total;
    const float excl = __shfl_up(inc, 1);
    float run = wbase + (lane ? excl : 0.f);
    int cand = 0x7fffffff, last_pos = -1;
    for (int v = v0; v < v1 && cand == 0x7fffffff; v += 4 * SAMPLE_BATCH) {
        float4 pv[SAMPLE_BATCH];
        load_batch(P, v, v1, 0.f, pv);
#pragma unroll
        for (int j = 0; j < SAMPLE_BATCH; ++j) {
            const float e[4] = {pv[j].x, pv[j].y, pv[j].z, pv[j].w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                if (cand == 0x7fffffff && e[k] > 0.f) {
                    last_pos = v + 4 * j + k;
                    run += e[k];
                    if (run > target) cand = last_pos;
                }
            }
        }
    }
    cand = block_reduce<2>(cand, ired);
    if (cand == 0x7fffffff)  // rounding left the target beyond the last prefix
        cand = block_reduce<1>(last_pos, ired);
    if (tid == 0) {
        for (int k = 0; k < n; ++k) a.acc->path[k] = path_s[k];
        a.acc->accept_len = n;
        a.acc->bonus = cand;
    }
}

// ---------------------------------------------------------------------------
// Large-M prefill: a prompt chunk of M tokens (padded to Mp, a multiple of
// 128) in one causal pass.  The projections are a dense contraction here, so
// they run on an MFMA GEMM over the packed weights of the verify path (block
// (k-step s, 16-row block gb) at (s NB + gb) 512) and split-layout
// activations of the whole chunk (MT = Mp / 16 token tiles), with the verify
// path's epilogues fused: rotary + K/V write, SwiGLU, residual + the next
// norm's input.  Every norm's 1/rms, a per-token scalar, is applied by its
// consumer's epilogue from sums of squares over 64-row slices (Mp x d / 64
// partials), so no fp32 GEMM output goes through HBM.

constexpr int PF_THREADS = 256;

// Embedding rows of the chunk: x = E[token], the first norm's numerator
// x * gain in split layout and the sums of squares of 64-column slices;
// tokens >= M get zeros.  One workgroup per token, 4 columns per thread.
__global__ __launch_bounds__(PF_THREADS) void k_pf_embed(const int32_t *tokens, const uint16_t *embed, int M, int d,
                                                         int MT, const uint16_t *gain, float *x, uint16_t *us,
                                                         float *ssq)
{
    const int m = blockIdx.x, nsq = d / 64;
    for (int k = 4 * threadIdx.x; k < d; k += 4 * PF_THREADS) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (m < M) {
            const uint2 e = *reinterpret_cast<const uint2 *>(embed + (size_t)tokens[m] * d + k);
            v = make_float4(__uint_as_float(e.x << 16), __uint_as_float(e.x & 0xffff0000u), __uint_as_float(e.y << 16),
                            __uint_as_float(e.y & 0xffff0000u));
        }
        *reinterpret_cast<float4 *>(x + (size_t)m * d + k) = v;
        store_split4(us, m, k, MT,
                     make_float4(v.x * bf2f(gain[k]), v.y * bf2f(gain[k + 1]), v.z * bf2f(gain[k + 2]),
                                 v.w * bf2f(gain[k + 3])));
        // 16 neighbouring threads hold one 64-column slice
        float ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, v.w * v.w)));
        ss += __shfl_xor(ss, 1);
        ss += __shfl_xor(ss, 2);
        ss += __shfl_xor(ss, 4);
        ss += __shfl_xor(ss, 8);
        if ((threadIdx.x & 15) == 0) ssq[(size_t)m * nsq + k / 64] = ss;
    }
}

// The prefill GEMM.  Workgroup = NWR x NWT waves over 64 NWR rows (4 blocks
// per wave) x 16 TT NWT tokens (TT token tiles per wave).  Per k-step each
// wave loads its 4 weight blocks into registers, the workgroup stages the
// activation slab of its token tiles (hi + lo) in LDS, and each wave runs
// 8 TT MFMAs (16x16x32 bf16, hi and lo into the same accumulator).  A
// wave's loads return in order, so weights and activations share one lead
// of LEAD k-steps (activations first in each step's loads).  With BPRE the
// slab is stashed two k-steps ahead into three LDS buffers and each wave
// reads its B operands one k-step ahead into registers; without it the slab
// is stashed one k-step ahead into two buffers and read just before use.
template <int EPI, int NWR, int NWT, int TT, int LEAD, bool BPRE>
__global__ __launch_bounds__(64 * NWR * NWT) void k_pf_gemm(PfArgs a)
{
    constexpr int NW = NWR * NWT, NT = 64 * NW, BW = 4, XT = NWT * TT, NBUF = BPRE ? 3 : 2;
    // the activation slab of a k-step: XE u32x4 (hi + lo of XT token
    // tiles), XL of them staged per thread (whole waves idle past XE)
    constexpr int XE = XT * 2 * 64, XL = (XE + NT - 1) / NT;
    static_assert(LEAD >= (BPRE ? 3 : 2), "the stash needs its loads a k-step earlier");
    // k-steps per unrolled round: register slots (st % LEAD) and B register
    // sets (st % 2) are compile-time in it
    constexpr int UR = (BPRE && LEAD % 2) ? 2 * LEAD : LEAD;
    __shared__ u32x4 xsm[NBUF][XT * 2 * 64];
    __shared__ float rinv_s[16 * XT];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, tid = threadIdx.x;
    const int wr = wave % NWR, wt = wave / NWR;
    // 1-D grid, XCD-aware: workgroups are dispatched to the 8 XCDs round
    // robin (workgroup b to XCD b % 8, 32 CUs each), so XCD x takes tiles
    // [x per, (x + 1) per) of the row-tile-major order: every XCD gets the
    // same count, and the token groups of a row tile share one XCD's L2 for
    // the row tile's weights (at most two XCDs at a chunk boundary).  Token
    // groups of XT tiles; the last one may be short (its missing tiles
    // re-read the last token tile and are never stored).
    const int n_tt = (a.MT + XT - 1) / XT, n_rt = (a.NB + NWR * BW - 1) / (NWR * BW);
    const int n_tiles = n_rt * n_tt, per = (n_tiles + 7) / 8;
    const int L = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
    if (L >= n_tiles) return;  // padding of the grid to 8 x per
    const int rtile = L / n_tt;
    const int tt0 = (L - rtile * n_tt) * XT;                 // first token tile of the workgroup
    const int gb0 = (rtile * NWR + wr) * BW;                 // first block of this wave
    const int S = a.K / 32;
    if (EPI != EPI_RESID) {
        for (int m = tid; m < 16 * min(XT, a.MT - tt0); m += NT) {
            const float *p = a.ssq_in + (size_t)(tt0 * 16 + m) * a.nsq_in;
            float sum = 0.f;
            for (int c = 0; c < a.nsq_in; ++c) sum += p[c];
            rinv_s[m] = 1.0f / sqrtf(sum / (float)a.d + a.eps);
        }
    }
    // buffer loads: the per-lane byte offsets stay fixed, a scalar offset moves
    // by one k-step (so no address register is rewritten while a load into a
    // neighbouring register is in flight); blocks past NB re-read the last
    // block (their sums are dropped)
    const __amdgpu_buffer_rsrc_t rw = rsrc_of(a.packed), rx = rsrc_of(a.xs);
    uint32_t wofs[BW], xofs[XL];
#pragma unroll
    for (int b = 0; b < BW; ++b) wofs[b] = (uint32_t)(min(gb0 + b, a.NB - 1) * 1024 + lane * 16);
#pragma unroll
    for (int i = 0; i < XL; ++i) {
        const int e = min(tid + NT * i, XE - 1), tile = min(tt0 + e / 128, a.MT - 1);
        xofs[i] = (uint32_t)((tile * 128 + e % 128) * 16);
    }
    const uint32_t wstep = (uint32_t)a.NB * 1024u, xstep = (uint32_t)a.MT * 2048u;
    u32x4 wb[LEAD][BW], stg[LEAD][XL];
    auto fetch = [&](int j, int st) {
#pragma unroll
        for (int i = 0; i < XL; ++i)
            stg[j][i] = __builtin_amdgcn_raw_buffer_load_b128(rx, xofs[i], (uint32_t)st * xstep, 0);
#pragma unroll
        for (int b = 0; b < BW; ++b)
            wb[j][b] = __builtin_amdgcn_raw_buffer_load_b128(rw, wofs[b], (uint32_t)st * wstep, DV_NT);
    };
    auto stash = [&](int j, int buf) {
#pragma unroll
        for (int i = 0; i < XL; ++i)
            if (XE % NT == 0 || tid + NT * i < XE) xsm[buf][tid + NT * i] = stg[j][i];
    };
    f32x4 acc[BW][TT];
#pragma unroll
    for (int b = 0; b < BW; ++b)
#pragma unroll
        for (int t = 0; t < TT; ++t) acc[b][t] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto mma = [&](int j, int t, const u32x4 &hv, const u32x4 &lv) {
        const bf16x8 hi = __builtin_bit_cast(bf16x8, hv), lo = __builtin_bit_cast(bf16x8, lv);
#pragma unroll
        for (int b = 0; b < BW; ++b) {
            const bf16x8 w = __builtin_bit_cast(bf16x8, wb[j][b]);
            acc[b][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, hi, acc[b][t], 0, 0, 0);
            acc[b][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, lo, acc[b][t], 0, 0, 0);
        }
    };
    auto xat = [&](int buf, int t, int q) -> u32x4 { return xsm[buf][((wt * TT + t) * 2 + q) * 64 + lane]; };
    // Loads and stashes are issued unconditionally (k-steps past the end
    // re-read the last one and are never used), so the number of loads in
    // flight behind each one is the same on every path and every wait is the
    // one the pipeline needs.  K-step st: weights in register slot st % LEAD.
#pragma unroll
    for (int j = 0; j < LEAD; ++j) fetch(j, min(j, S - 1));
    if constexpr (BPRE) {
        // activations in LDS buffer st % 3, stashed two k-steps ahead; B
        // operands in register set st % 2, read one k-step ahead.  The
        // barrier after step st makes step st + 2's stash visible, and every
        // read of buffer (st + 3) % 3 (step st's operands, read in step
        // st - 1) is done before step st + 1 overwrites it.
        u32x4 xb[2][TT][2];
        auto bread = [&](int r, int buf) {
#pragma unroll
            for (int t = 0; t < TT; ++t)
#pragma unroll
                for (int q = 0; q < 2; ++q) xb[r][t][q] = xat(buf, t, q);
        };
        stash(0, 0);
        stash(1, 1);
        __syncthreads();
        bread(0, 0);
        for (int s0 = 0; s0 < S; s0 += UR) {
#pragma unroll
            for (int u = 0; u < UR; ++u) {
                const int st = s0 + u, j = u % LEAD;
                if (st < S) {
#pragma unroll
                    for (int t = 0; t < TT; ++t) mma(j, t, xb[u & 1][t][0], xb[u & 1][t][1]);
                }
                bread((u + 1) & 1, (st + 1) % 3);
                stash((u + 2) % LEAD, (st + 2) % 3);
                fetch(j, min(st + LEAD, S - 1));
                __syncthreads();
            }
        }
    } else {
        // activations in LDS buffer st % 2, stashed one k-step ahead; the
        // barrier after step st makes step st + 1's stash visible, and every
        // read of buffer st % 2 is done before step st + 1 overwrites it
        stash(0, 0);
        __syncthreads();
        for (int s0 = 0; s0 < S; s0 += UR) {
#pragma unroll
            for (int u = 0; u < UR; ++u) {
                const int st = s0 + u, j = u % LEAD;
                if (st < S) {
#pragma unroll
                    for (int t = 0; t < TT; ++t) mma(j, t, xat(st & 1, t, 0), xat(st & 1, t, 1));
                }
                stash((u + 1) % LEAD, (st + 1) & 1);
                fetch(j, min(st + LEAD, S - 1));
                __syncthreads();
            }
        }
    }

    // ---- epilogues: lane l holds rows 4 (l / 16) + jj of block gb0 + b for
    // token (tt0 + wt TT + t) 16 + l % 16
    const int n16 = lane & 15, r4 = 4 * (lane >> 4);
    if (EPI == EPI_QKV) {
        const int per_seg = a.d / DV_GEMM_TILE, per_head = a.hd / DV_GEMM_TILE, half = a.hd / 2;
#pragma unroll
        for (int p = 0; p < BW / 2; ++p) {
            const int gb = gb0 + 2 * p;
            if (gb >= a.NB) break;
            const int tile = gb >> 1, seg = tile / per_seg, tt = tile - seg * per_seg;
            const int h = tt / per_head, j0 = (tt - h * per_head) * 16 + r4;
#pragma unroll
            for (int t = 0; t < TT; ++t) {
                const int ml = (wt * TT + t) * 16 + n16, m = tt0 * 16 + ml;
                if (m >= a.M) continue;
                const float ri = rinv_s[ml];
                float y1[4], y2[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    y1[jj] = acc[2 * p][t][jj] * ri;
                    y2[jj] = acc[2 * p + 1][t][jj] * ri;
                }
                const int pos = a.P0 + m;
                if (seg < 2) {
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        const float c = a.rope_cos[(size_t)pos * half + j0 + jj];
                        const float sn = a.rope_sin[(size_t)pos * half + j0 + jj];
                        const float o1 = y1[jj] * c - y2[jj] * sn, o2 = y2[jj] * c + y1[jj] * sn;
                        y1[jj] = o1;
                        y2[jj] = o2;
                    }
                }
                if (seg == 0) {
                    float *qr = a.q + (size_t)m * a.d + h * a.hd + j0;
                    *reinterpret_cast<float4 *>(qr) = make_float4(y1[0], y1[1], y1[2], y1[3]);
                    *reinterpret_cast<float4 *>(qr + half) = make_float4(y2[0], y2[1], y2[2], y2[3]);
                } else if (seg == 1) {  // K: [H][cap][hd]
                    uint16_t *kr = reinterpret_cast<uint16_t *>(a.kc) + ((size_t)h * a.cap + pos) * a.hd + j0;
                    *reinterpret_cast<uint2 *>(kr) = make_uint2(f2bf(y1[0]) | (uint32_t)f2bf(y1[1]) << 16,
                                                                f2bf(y1[2]) | (uint32_t)f2bf(y1[3]) << 16);
                    *reinterpret_cast<uint2 *>(kr + half) = make_uint2(f2bf(y2[0]) | (uint32_t)f2bf(y2[1]) << 16,
                                                                       f2bf(y2[2]) | (uint32_t)f2bf(y2[3]) << 16);
                } else {                // V: [H][cap/32][hd][32]
                    uint16_t *vh = reinterpret_cast<uint16_t *>(a.vc) + (size_t)h * a.hd * a.cap;
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        vh[v_index(j0 + jj, pos, a.hd)] = f2bf(y1[jj]);
                        vh[v_index(j0 + jj + half, pos, a.hd)] = f2bf(y2[jj]);
                    }
                }
            }
        }
    } else if (EPI == EPI_SWIGLU) {
        // gate block 2p and up block 2p + 1 hold h columns 16 (gb / 2) + ...
#pragma unroll
        for (int p = 0; p < BW / 2; ++p) {
            const int gb = gb0 + 2 * p;
            if (gb >= a.NB) break;
            const int f0 = 16 * (gb >> 1) + r4;
#pragma unroll
            for (int t = 0; t < TT; ++t) {
                if (tt0 + wt * TT + t >= a.MT) break;  // a short last token group
                const int ml = (wt * TT + t) * 16 + n16, m = tt0 * 16 + ml;
                float hv[4] = {0.f, 0.f, 0.f, 0.f};
                if (m < a.M) {
                    const float ri = rinv_s[ml];
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) hv[jj] = silu(acc[2 * p][t][jj] * ri) * (acc[2 * p + 1][t][jj] * ri);
                }
                store_split4(a.hs, m, f0, a.MT, make_float4(hv[0], hv[1], hv[2], hv[3]));
            }
        }
    } else {  // EPI_RESID
        if (gb0 < a.NB) {
            const int nsq = a.d / 64;
#pragma unroll
            for (int t = 0; t < TT; ++t) {
                if (tt0 + wt * TT + t >= a.MT) break;  // a short last token group (wave-uniform)
                const int ml = (wt * TT + t) * 16 + n16, m = tt0 * 16 + ml;
                float ss = 0.f;
#pragma unroll
                for (int b = 0; b < BW; ++b) {
                    const int r = 16 * (gb0 + b) + r4;
                    float4 xv = make_float4(0.f, 0.f, 0.f, 0.f);
                    if (m < a.M) {
                        float *xp = a.x + (size_t)m * a.d + r;
                        xv = *reinterpret_cast<const float4 *>(xp);
                        xv.x += acc[b][t][0];
                        xv.y += acc[b][t][1];
                        xv.z += acc[b][t][2];
                        xv.w += acc[b][t][3];
                        *reinterpret_cast<float4 *>(xp) = xv;
                    }
                    ss = fmaf(xv.x, xv.x, fmaf(xv.y, xv.y, fmaf(xv.z, xv.z, fmaf(xv.w, xv.w, ss))));
                    store_split4(a.us, m, r, a.MT,
                                 make_float4(xv.x * bf2f(a.gain[r]), xv.y * bf2f(a.gain[r + 1]),
                                             xv.z * bf2f(a.gain[r + 2]), xv.w * bf2f(a.gain[r + 3])));
                }
                ss += __shfl_xor(ss, 16);
                ss += __shfl_xor(ss, 32);
                if (lane < 16) a.ssq_out[(size_t)m * nsq + gb0 / 4] = ss;
            }
        }
    }
}

// Causal attention of the chunk's queries (positions P0 + i) over cache slots
// [0, P0 + i].  Workgroup = 64 queries of one head, each wave 16 of them; the
// workgroup stages every 32-key tile up to its last query in LDS once (K rows
// and the tile's V block, rows padded against bank conflicts; the next tile's
// global loads are in flight while the current one is used), and each wave
// uses the tiles up to its own last query.  The scores and the running
// softmax follow the tree-attention kernel (MFMA with q split in hi + lo,
// exp2 in log2 units); the output goes to the O projection's operand (split
// layout of MT token tiles).  Grid (heads, query blocks) with the last query
// block first: workgroups are dispatched in order, so the longest ones (the
// most keys) start first and the short ones fill in behind them.
template <int HD>
__global__ __launch_bounds__(256) void k_attn_causal(const float *q, const uint16_t *kc_l, const uint16_t *vc_l,
                                                     int M, int P0, int H, int cap, int MT, uint16_t *out)
{
    constexpr int NC = HD / 32, ND = HD / 16;
    constexpr int KROW = HD * 2 + 16;          // bytes per staged key row (padded)
    constexpr int VROW = 80;                   // bytes per staged dim row of 32 values (padded)
    constexpr int KBYTES = 32 * KROW, VBYTES = HD * VROW;
    constexpr int KCH = 32 * HD / 8, VCH = HD * 4;  // 16-byte chunks of a tile's K and V
    constexpr int CPT = (KCH + VCH + 255) / 256;     // chunks per thread
    __shared__ __align__(16) unsigned char smem[2][KBYTES + VBYTES];
    const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = lane & 15, g = lane >> 4;
    const int q0 = (gridDim.y - 1 - blockIdx.y) * 64;
    const int qb = q0 + wave * 16;               // first query of this wave
    const int D = H * HD;
    const int kend_wg = P0 + min(q0 + 64, M);    // keys the workgroup may see
    const int ntile = (kend_wg + 31) / 32;
    const bool active = qb < M;
    const int kend = P0 + min(qb + 16, M);       // keys this wave may see
    const int wtiles = active ? (kend + 31) / 32 : 0;
    const float scale2 = 1.4426950408889634f / sqrtf((float)HD);
    const uint16_t *kc = kc_l + (size_t)h * cap * HD;
    const uint16_t *vc = vc_l + (size_t)h * HD * cap;
    const int qi = min(qb + n, M - 1);          // this lane's query (B operand column)
    const int lim = P0 + qb + n;                // last key it sees

    bf16x8 qh[NC], ql[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const float *qp = q + (size_t)qi * D + h * HD + 32 * c + 8 * g;
        split_hi_lo(*reinterpret_cast<const float4 *>(qp), *reinterpret_cast<const float4 *>(qp + 4), qh[c], ql[c]);
    }
    // global -> registers -> LDS staging of tile t: chunk e < KCH is 16 bytes
    // of key row e / (HD / 8) (rows past the workgroup's last key repeat it),
    // the rest 16 bytes of the tile's V block (dim row, 8 slots)
    u32x4 stg[CPT];
    auto fetch = [&](int t) {
        const int k0 = 32 * t;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int e = tid + 256 * i;
            if (e < KCH) {
                const int r = e / (HD / 8), c8 = e % (HD / 8);
                const int key = min(k0 + r, kend_wg - 1);
                stg[i] = *reinterpret_cast<const u32x4 *>(kc + (size_t)key * HD + 8 * c8);
            } else if (e < KCH + VCH) {
                const int ev = e - KCH;
                stg[i] = *reinterpret_cast<const u32x4 *>(vc + (size_t)(k0 >> 5) * HD * 32 + 8 * ev);
            }
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int e = tid + 256 * i;
            if (e < KCH) {
                const int r = e / (HD / 8), c8 = e % (HD / 8);
                *reinterpret_cast<u32x4 *>(&smem[buf][r * KROW + 16 * c8]) = stg[i];
            } else if (e < KCH + VCH) {
                const int ev = e - KCH, dr = ev >> 2, c8 = ev & 3;
                *reinterpret_cast<u32x4 *>(&smem[buf][KBYTES + dr * VROW + 16 * c8]) = stg[i];
            }
        }
    };

    float m_run = -INFINITY, l_run = 0.f;
    f32x4 o[ND];
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) o[dt] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto process = [&](int t, int buf) {
        const int k0 = 32 * t;
        const unsigned char *ks = smem[buf], *vs = smem[buf] + KBYTES;
        const int ra = 8 * (n >> 2) + (n & 3), rb = ra + 4;
        f32x4 sa = (f32x4){0.f, 0.f, 0.f, 0.f}, sb = sa;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const bf16x8 ka8 = *reinterpret_cast<const bf16x8 *>(ks + ra * KROW + 64 * c + 16 * g);
            const bf16x8 kb8 = *reinterpret_cast<const bf16x8 *>(ks + rb * KROW + 64 * c + 16 * g);
            sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka8, qh[c], sa, 0, 0, 0);
            sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb8, qh[c], sb, 0, 0, 0);
            sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka8, ql[c], sa, 0, 0, 0);
            sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb8, ql[c], sb, 0, 0, 0);
        }
        // scores of query (lane n) for keys k0 + 8g + i
        float sv[8], mt = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int key = k0 + 8 * g + i;
            const float sc = (i < 4 ? sa[i] : sb[i - 4]) * scale2;
            sv[i] = key <= lim ? sc : -INFINITY;
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
        float al[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) al[j] = __shfl(alpha, 4 * g + j);
        u32x4 vt[ND];
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
            vt[dt] = *reinterpret_cast<const u32x4 *>(vs + (dt * 16 + n) * VROW + 16 * g);
        if (k0 + 32 > kend) {
            // slots past the wave's last key hold nothing of this chunk yet
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int key = k0 + 8 * g + 2 * w;
                    uint32_t x = vt[dt][w];
                    if (key >= kend) x &= 0xffff0000u;
                    if (key + 1 >= kend) x &= 0x0000ffffu;
                    vt[dt][w] = x;
                }
        }
        bf16x8 ph, pl;
        split_hi_lo(make_float4(pv[0], pv[1], pv[2], pv[3]), make_float4(pv[4], pv[5], pv[6], pv[7]), ph, pl);
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
#pragma unroll
            for (int j = 0; j < 4; ++j) o[dt][j] *= al[j];
            const bf16x8 v8 = __builtin_bit_cast(bf16x8, vt[dt]);
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, v8, o[dt], 0, 0, 0);
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, v8, o[dt], 0, 0, 0);
        }
    };
    fetch(0);
    stash(0);
    __syncthreads();
    for (int t = 0; t < ntile; ++t) {
        const int buf = t & 1;
        if (t + 1 < ntile) fetch(t + 1);  // in flight while tile t is used
        if (t < wtiles) process(t, buf);
        if (t + 1 < ntile) stash(buf ^ 1);
        __syncthreads();
    }
    if (!active) return;
    // rows of o are queries qb + 4g + j; their sums l sit in lanes 4g + j
    float lr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) lr[j] = __shfl(l_run, 4 * g + j);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int i = qb + 4 * g + j;
        if (i >= M) continue;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) store_split(out, i, h * HD + dt * 16 + n, MT, o[dt][j] / lr[j]);
    }
}

// ---------------------------------------------------------------------------
// Draft side.  Dynamic Gated Fusion around three weight-streaming
// projections (k_proj with the plain-output epilogue, split-layout operands):
//   prep: parent features and token embeddings -> split-layout operands
//   mid:  h1 = W_h f, h2 = W_e e -> split-layout operand of [h1 || h2]
//   out:  g = sigmoid(W_g [h1 || h2]); x0 = g h1 + (1 - g) h2
// DGF operands in split layout (the projection kernel's B operand), one
// workgroup per token row m < Mpad: feature rows and the token embeddings
// (bf16, so exact: lo = 0); rows n..Mpad are zero.
__global__ __launch_bounds__(PF_THREADS) void k_dgf_in(const float *feat, const uint16_t *embed, DgfTokens t, int n,
                                                       int d, int MT, uint16_t *xf, uint16_t *xe)
{
    const int m = blockIdx.x;
    for (int k = 4 * threadIdx.x; k < d; k += 4 * PF_THREADS) {
        float4 f = make_float4(0.f, 0.f, 0.f, 0.f), e = f;
        if (m < n) {
            f = *reinterpret_cast<const float4 *>(feat + (size_t)m * d + k);
            const uint2 eb = *reinterpret_cast<const uint2 *>(embed + (size_t)t.tok[m] * d + k);
            e = make_float4(bf2f(eb.x & 0xffffu), bf2f(eb.x >> 16), bf2f(eb.y & 0xffffu), bf2f(eb.y >> 16));
        }
        store_split4(xf, m, k, MT, f);
        store_split4(xe, m, k, MT, e);
    }
}

// gate input [h1 || h2] (K = 2 d) in split layout
__global__ __launch_bounds__(PF_THREADS) void k_dgf_gate_in(const float *h1, const float *h2, int n, int d, int MT,
                                                            uint16_t *xg)
{
    const int m = blockIdx.x;
    for (int k = 4 * threadIdx.x; k < d; k += 4 * PF_THREADS) {
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
        if (m < n) {
            a = *reinterpret_cast<const float4 *>(h1 + (size_t)m * d + k);
            b = *reinterpret_cast<const float4 *>(h2 + (size_t)m * d + k);
        }
        store_split4(xg, m, k, MT, a);
        store_split4(xg, m, d + k, MT, b);
    }
}

// x0 = g h1 + (1 - g) h2, g = sigmoid(z)
__global__ __launch_bounds__(PF_THREADS) void k_dgf_mix(const float *z, const float *h1, const float *h2, int d,
                                                        float *x0)
{
    const int i = blockIdx.x;
    for (int k = threadIdx.x; k < d; k += PF_THREADS) {
        const size_t o = (size_t)i * d + k;
        const float g = 1.f / (1.f + expf(-z[o]));
        x0[o] = g * h1[o] + (1.f - g) * h2[o];
    }
}

// Row gather: dst[r] = src[idx[r]] (feature rows of d floats).
__global__ __launch_bounds__(PF_THREADS) void k_gather_rows(const float *src, RowIndex ix, int d, float *dst)
{
    const int r = blockIdx.x;
    const float *sp = src + (size_t)ix.idx[r] * d;
    for (int k = 4 * threadIdx.x; k < d; k += 4 * PF_THREADS)
        *reinterpret_cast<float4 *>(dst + (size_t)r * d + k) = *reinterpret_cast<const float4 *>(sp + k);
}

// The `k` most probable tokens of logits row rows[b] (one workgroup per row):
// p = softmax(z) in fp32 (max, then the sum of exp in a fixed order), then k
// rounds of a block-wide arg-max over the ids not taken yet (larger p, then
// lower id).  V <= 32 * 1024.
__global__ __launch_bounds__(1024) void k_topk_probs(const float *logits, int V, TopkArgs a)
{
    __shared__ float red[16];
    __shared__ float bv[16];
    __shared__ int bi[16];
    __shared__ int win;
    const int tid = threadIdx.x;
    const float *z = logits + (size_t)a.rows[blockIdx.x] * V;
    float zv[32];
    float mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        const int v = tid + 1024 * c;
        zv[c] = v < V ? z[v] : -INFINITY;
        mx = fmaxf(mx, zv[c]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    mx = red[0];
    for (int w = 1; w < 16; ++w) mx = fmaxf(mx, red[w]);
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < 32; ++c) {
        zv[c] = zv[c] == -INFINITY ? 0.f : expf(zv[c] - mx);
        sum += zv[c];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
    __syncthreads();
    if ((tid & 63) == 0) red[tid >> 6] = sum;
    __syncthreads();
    float tot = 0.f;
    for (int w = 0; w < 16; ++w) tot += red[w];
    uint32_t taken = 0;
    for (int r = 0; r < a.k; ++r) {
        float best = -1.f;
        int bid = 0x7fffffff;
#pragma unroll
        for (int c = 0; c < 32; ++c) {
            const int v = tid + 1024 * c;
            if (v < V && !((taken >> c) & 1u) && zv[c] > best) { best = zv[c]; bid = v; }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const float v2 = __shfl_xor(best, off);
            const int i2 = __shfl_xor(bid, off);
            arg_better(best, bid, v2, i2);
        }
        if ((tid & 63) == 0) {
            bv[tid >> 6] = best;
            bi[tid >> 6] = bid;
        }
        __syncthreads();
        if (tid == 0) {
            float b = bv[0];
            int id = bi[0];
            for (int w = 1; w < 16; ++w) arg_better(b, id, bv[w], bi[w]);
            win = id;
            a.out_tok[blockIdx.x * DV_TOPK_MAX + r] = id;
            a.out_p[blockIdx.x * DV_TOPK_MAX + r] = b / tot;
        }
        __syncthreads();
        if (win % 1024 == tid) taken |= 1u << (win / 1024);
    }
}

// ---------------------------------------------------------------------------
// KV commit: slot P+k <- slot P+path[k] for k < n, for every (layer, head)
// of K (blockIdx.y = 0, rows [cap][hd]) and V (1, entries at v_index).  A
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
        const size_t src = is_v ? v_index(d, a.P + a.path[k], a.hd) : (size_t)(a.P + a.path[k]) * a.hd + d;
        buf[e] = base[src];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < nel; e += blockDim.x) {
        const int k = e / a.hd, d = e % a.hd;
        if (a.path[k] == k) continue;
        const size_t dst = is_v ? v_index(d, a.P + k, a.hd) : (size_t)(a.P + k) * a.hd + d;
        base[dst] = buf[e];
    }
}

// ---------------------------------------------------------------------------
// launchers

GemmShape gemm_shape(int rb) { return rb >= 4 ? GemmShape{4, 2} : GemmShape{4, 4}; }

// Waves per workgroup of the MFMA projection.  More than one token tile
// holds more accumulators and operands per wave, so each wave keeps fewer
// steps in flight; with bf16 weights 8 waves (two per SIMD) then keep the
// loads coming (int8 weights: 4, their dequantisation registers would spill).
static int proj_waves(int wkind, int mt, int rb) { return mt >= 2 && wkind == W_BF16 ? 8 : gemm_shape(rb).nw; }

template <int EPI, typename KV, int RB, bool Q8>
static const void *proj_kernel_mt(int mt)
{
    constexpr int U1 = RB >= 4 ? 2 : 4, NWM = Q8 ? 4 : 8;
    if constexpr (RB == 8) {
        // 8-block groups: one token tile at most (see gemm_rb8)
        if (mt == 0) return (const void *)k_proj<0, EPI, KV, 4, U1, RB, Q8>;
        if (mt == 1) return (const void *)k_proj<1, EPI, KV, 4, U1, RB, Q8>;
        return nullptr;
    } else {
        switch (mt) {
        case 0: return (const void *)k_proj<0, EPI, KV, 4, U1, RB, Q8>;  // half split layout
        case 1: return (const void *)k_proj<1, EPI, KV, 4, U1, RB, Q8>;
        case 2: return (const void *)k_proj<2, EPI, KV, NWM, 2, RB, Q8>;
        case 3: return (const void *)k_proj<3, EPI, KV, NWM, 2, RB, Q8>;
        case 4: return (const void *)k_proj<4, EPI, KV, NWM, 2, RB, Q8>;
        default: return nullptr;
        }
    }
}

template <int EPI>
static const void *gemm_kernel(int wkind, int use_mfma, int mt, int rb)
{
    if constexpr (EPI == EPI_PLAIN) {  // bf16 weights, MFMA path only
        if (wkind != W_BF16 || !use_mfma) return nullptr;
        if (rb == 4) return proj_kernel_mt<EPI, uint16_t, 4, false>(mt);
        if (rb == 2) return proj_kernel_mt<EPI, uint16_t, 2, false>(mt);
        return nullptr;
    } else {
        if (wkind != W_F32 && use_mfma) {
            const bool q8 = wkind == W_I8;
            if constexpr (EPI == EPI_SWIGLU) {
                if (rb == 8) return q8 ? proj_kernel_mt<EPI, uint16_t, 8, true>(mt) : proj_kernel_mt<EPI, uint16_t, 8, false>(mt);
            }
            if constexpr (EPI == EPI_LOGITS) {  // bf16 lm_head measured slower in 8-block groups
                if (rb == 8 && q8) return proj_kernel_mt<EPI, uint16_t, 8, true>(mt);
            }
            if (rb == 8) return nullptr;
            if (rb == 4) return q8 ? proj_kernel_mt<EPI, uint16_t, 4, true>(mt) : proj_kernel_mt<EPI, uint16_t, 4, false>(mt);
            if (rb == 2) return q8 ? proj_kernel_mt<EPI, uint16_t, 2, true>(mt) : proj_kernel_mt<EPI, uint16_t, 2, false>(mt);
            return nullptr;
        }
        if (wkind == W_BF16) return (const void *)k_gemm_valu<uint16_t, EPI, uint16_t>;
        if (wkind == W_F32) return (const void *)k_gemm_valu<float, EPI, float>;
        return nullptr;  // int8 weights have no VALU kernel
    }
}

static const void *gemm_kernel_any(int epi, int wkind, int use_mfma, int mt, int rb)
{
    switch (epi) {
    case EPI_QKV: return gemm_kernel<EPI_QKV>(wkind, use_mfma, mt, rb);
    case EPI_RESID: return gemm_kernel<EPI_RESID>(wkind, use_mfma, mt, rb);
    case EPI_SWIGLU: return gemm_kernel<EPI_SWIGLU>(wkind, use_mfma, mt, rb);
    case EPI_LOGITS: return gemm_kernel<EPI_LOGITS>(wkind, use_mfma, mt, rb);
    case EPI_PLAIN: return gemm_kernel<EPI_PLAIN>(wkind, use_mfma, mt, rb);
    }
    return nullptr;
}

static int gemm_threads(int wkind, int use_mfma, int mt, int rb)
{
    return (wkind != W_F32 && use_mfma) ? 64 * proj_waves(wkind, mt, rb) : 256;
}

int gemm_blocks_per_cu(int epi, int wkind, int use_mfma, int mt, int rb)
{
    static int cache[5][3][2][5][3];
    if (wkind < 0 || wkind > 2 || epi < 0 || epi > 4) return 1;
    if (mt < 0 || mt > 4) return 1;
    int &c = cache[epi][wkind][use_mfma ? 1 : 0][mt][rb == 8 ? 2 : (rb == 4 ? 1 : 0)];
    if (c == 0) {
        const void *k = gemm_kernel_any(epi, wkind, use_mfma, mt, rb);
        int n = 0;
        if (!k || hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, gemm_threads(wkind, use_mfma, mt, rb), 0) !=
                      hipSuccess || n < 1)
            n = 1;
        c = n;
    }
    return c;
}

bool gemm_has_rb8(int epi, int wkind, int mt) { return gemm_kernel_any(epi, wkind, 1, mt, 8) != nullptr; }

hipError_t launch_gemm(const GemmArgs &a, int grid, int epi, int wkind, int use_mfma, hipStream_t s,
                       hipEvent_t ev_start, hipEvent_t ev_stop)
{
    const int mt = a.half ? 0 : a.Mpad / 16;
    if (a.half && a.M > 8) return hipErrorInvalidValue;
    const void *k = gemm_kernel_any(epi, wkind, use_mfma, mt, a.rb);
    if (!k || grid < 1) return hipErrorInvalidValue;
    if (wkind == W_I8 && (!a.scale || a.K % 64)) return hipErrorInvalidValue;
    GemmArgs arg = a;
    void *params[] = {&arg};
    const dim3 block(gemm_threads(wkind, use_mfma, mt, a.rb));
    // with events: timestamps taken by the dispatch itself (no extra packets)
    if (ev_start && ev_stop) return hipExtLaunchKernel(k, dim3(grid), block, params, 0, s, ev_start, ev_stop, 0);
    return hipLaunchKernel(k, dim3(grid), block, params, 0, s);
}

hipError_t launch_pack(const GemmArgs &a, int epi, int wkind, void *dst, hipStream_t s)
{
    if (a.rb != 2 && a.rb != 4) return hipErrorInvalidValue;
    if (wkind == W_I8) {
        if (a.K % 64) return hipErrorInvalidValue;
        hipLaunchKernelGGL(k_pack_blocks_i8, dim3(a.n_groups * a.rb, std::min(a.K / 64, 64)), dim3(64), 0, s, a, epi,
                           static_cast<uint8_t *>(dst));
    } else if (wkind == W_BF16) {
        hipLaunchKernelGGL(k_pack_blocks, dim3(a.n_groups * a.rb, std::min(a.K / 32, 64)), dim3(64), 0, s, a, epi,
                           static_cast<uint16_t *>(dst));
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_pack_scales(const GemmArgs &a, int epi, float *dst, hipStream_t s)
{
    if (a.rb != 2 && a.rb != 4) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pack_scales, dim3(a.n_groups * a.rb), dim3(16), 0, s, a, epi, dst);
    return hipGetLastError();
}

template <typename W>
static hipError_t embed_norm_dispatch(const NormArgs &a, int Mpad, hipStream_t s)
{
    const int slice = a.d / DV_NORM_SLICES;
    if (a.d % (4 * DV_NORM_SLICES)) return hipErrorInvalidValue;
    const dim3 grid(Mpad, DV_NORM_SLICES), block(DV_NORM_THREADS);
    switch ((slice + 4 * DV_NORM_THREADS - 1) / (4 * DV_NORM_THREADS)) {
    case 1: hipLaunchKernelGGL((k_embed_norm<W, 1>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_embed_norm<W, 2>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_embed_norm(const NormArgs &a, int Mpad, int weight_bf16, hipStream_t s)
{
    return weight_bf16 ? embed_norm_dispatch<uint16_t>(a, Mpad, s) : embed_norm_dispatch<float>(a, Mpad, s);
}

hipError_t launch_attention(const AttnArgs &a, int kv_bf16, hipStream_t s)
{
    const dim3 grid(a.n_split, a.H), block(256);
    // up to 8 key tiles per split: 8 waves holding one tile each; longer
    // splits: 4 waves with two tiles in flight each (one query tile) or one
    // each (more)
    const bool short_split = a.keys_per_split <= 8 * DV_ATTN_TILE;
    const dim3 b8(512), b4(256);
    // more than 16 nodes: every key tile serves all query tiles, with the
    // per-tile outputs in registers
    const int qt = a.tm.Mpad / 16;
    if (qt < 1 || qt > 4) return hipErrorInvalidValue;
    if (!kv_bf16) {
        if (a.hd == 128) hipLaunchKernelGGL(k_attn_f32<128>, grid, block, 0, s, a);
        else if (a.hd == 64) hipLaunchKernelGGL(k_attn_f32<64>, grid, block, 0, s, a);
        else return hipErrorInvalidValue;
        return hipGetLastError();
    }
    if (a.hd == 128) {
        if (short_split) {
            if (qt == 1) hipLaunchKernelGGL((k_attn_mfma<128, 8, false, 1>), grid, b8, 0, s, a);
            else if (qt == 2) hipLaunchKernelGGL((k_attn_mfma<128, 8, false, 2>), grid, b8, 0, s, a);
            else if (qt == 3) hipLaunchKernelGGL((k_attn_mfma<128, 8, false, 3>), grid, b8, 0, s, a);
            else hipLaunchKernelGGL((k_attn_mfma<128, 8, false, 4>), grid, b8, 0, s, a);
        } else if (qt == 1) hipLaunchKernelGGL((k_attn_mfma<128, 4, true, 1>), grid, b4, 0, s, a);
        else if (qt == 2) hipLaunchKernelGGL((k_attn_mfma<128, 4, false, 2>), grid, b4, 0, s, a);
        else if (qt == 3) hipLaunchKernelGGL((k_attn_mfma<128, 4, false, 3>), grid, b4, 0, s, a);
        else hipLaunchKernelGGL((k_attn_mfma<128, 4, false, 4>), grid, b4, 0, s, a);
    } else if (a.hd == 64) {
        if (short_split) {
            if (qt == 1) hipLaunchKernelGGL((k_attn_mfma<64, 8, false, 1>), grid, b8, 0, s, a);
            else if (qt == 2) hipLaunchKernelGGL((k_attn_mfma<64, 8, false, 2>), grid, b8, 0, s, a);
            else if (qt == 3) hipLaunchKernelGGL((k_attn_mfma<64, 8, false, 3>), grid, b8, 0, s, a);
            else hipLaunchKernelGGL((k_attn_mfma<64, 8, false, 4>), grid, b8, 0, s, a);
        } else if (qt == 1) hipLaunchKernelGGL((k_attn_mfma<64, 4, true, 1>), grid, b4, 0, s, a);
        else if (qt == 2) hipLaunchKernelGGL((k_attn_mfma<64, 4, false, 2>), grid, b4, 0, s, a);
        else if (qt == 3) hipLaunchKernelGGL((k_attn_mfma<64, 4, false, 3>), grid, b4, 0, s, a);
        else hipLaunchKernelGGL((k_attn_mfma<64, 4, false, 4>), grid, b4, 0, s, a);
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

hipError_t launch_accept_sampled(const SampleArgs &a, hipStream_t s)
{
    if (a.M < 1 || a.M > DV_TREE_MAX || a.V < 4 || a.V % 4) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_accept_sampled, dim3(1), dim3(SAMPLE_THREADS), 0, s, a);
    return hipGetLastError();
}

// Workspace of the allocation-free sampled acceptance (see dv.h,
// dv_accept_sampled_noalloc).  In host code `scratch` is only a stand-in for
// the symbol: its device address comes from hipGetSymbolAddress, once per
// device, and only that address is ever handed to a kernel or a copy.
static __device__ __align__(256) unsigned char scratch[DV_NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(void **out)
{
    static std::mutex mu;
    static void *addr[DV_NOALLOC_MAX_DEVICES];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= DV_NOALLOC_MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
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

hipError_t launch_pf_embed(const int32_t *tokens, const void *embed, int M, int Mp, int d, const void *gain, float *x,
                           uint16_t *us, float *ssq, hipStream_t s)
{
    if (d % 64 || Mp % 16 || M < 1 || M > Mp) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pf_embed, dim3(Mp), dim3(PF_THREADS), 0, s, tokens, static_cast<const uint16_t *>(embed), M, d,
                       Mp / 16, static_cast<const uint16_t *>(gain), x, us, ssq);
    return hipGetLastError();
}

#ifndef PF_CFG_MAIN
#define PF_CFG_MAIN 8, 1, 8, 4, false
#endif
#ifndef PF_CFG_RESID
#define PF_CFG_RESID 8, 1, 3, 4, true
#endif

template <int EPI, int NWR, int NWT, int TT, int LEAD, bool BPRE>
static hipError_t pf_launch(const PfArgs &a, hipStream_t s)
{
    constexpr int ROWS = 64 * NWR, XT = NWT * TT;
    // 1-D grid: 8 chunks of ceil(tiles / 8) (token groups x row tiles)
    const int n_rt = (a.NB * 16 + ROWS - 1) / ROWS, n_tiles = (a.MT + XT - 1) / XT * n_rt;
    const dim3 grid(8 * ((n_tiles + 7) / 8));
    hipLaunchKernelGGL((k_pf_gemm<EPI, NWR, NWT, TT, LEAD, BPRE>), grid, dim3(64 * NWR * NWT), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_pf_gemm(const PfArgs &a, int epi, hipStream_t s)
{
    if (a.K % 32 || a.NB < 1 || a.MT % 8 || a.d % 64 || a.M < 1 || a.M > 16 * a.MT) return hipErrorInvalidValue;
    if (epi == EPI_RESID) return pf_launch<EPI_RESID, PF_CFG_RESID>(a, s);
    if (epi == EPI_QKV) {
        if (a.hd != 64 && a.hd != 128) return hipErrorInvalidValue;
        return pf_launch<EPI_QKV, PF_CFG_MAIN>(a, s);
    }
    if (epi == EPI_SWIGLU) return pf_launch<EPI_SWIGLU, PF_CFG_MAIN>(a, s);
    return hipErrorInvalidValue;
}

hipError_t launch_attn_causal(const float *q, const void *kc, const void *vc, int M, int P0, int H, int hd, int cap,
                              int MT, uint16_t *out, hipStream_t s)
{
    const dim3 grid(H, (M + 63) / 64);
    const uint16_t *k16 = static_cast<const uint16_t *>(kc), *v16 = static_cast<const uint16_t *>(vc);
    if (hd == 128) hipLaunchKernelGGL(k_attn_causal<128>, grid, dim3(256), 0, s, q, k16, v16, M, P0, H, cap, MT, out);
    else if (hd == 64) hipLaunchKernelGGL(k_attn_causal<64>, grid, dim3(256), 0, s, q, k16, v16, M, P0, H, cap, MT, out);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_dgf_in(const float *feat, const void *embed, const DgfTokens &t, int n, int Mpad, int d,
                         uint16_t *xf, uint16_t *xe, hipStream_t s)
{
    if (n < 1 || n > Mpad || Mpad > DV_TREE_MAX || Mpad % 16 || d % 32) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_dgf_in, dim3(Mpad), dim3(PF_THREADS), 0, s, feat, static_cast<const uint16_t *>(embed), t, n, d,
                       Mpad / 16, xf, xe);
    return hipGetLastError();
}

hipError_t launch_dgf_gate_in(const float *h1, const float *h2, int n, int Mpad, int d, uint16_t *xg, hipStream_t s)
{
    if (n < 1 || n > Mpad || Mpad > DV_TREE_MAX || Mpad % 16 || d % 32) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_dgf_gate_in, dim3(Mpad), dim3(PF_THREADS), 0, s, h1, h2, n, d, Mpad / 16, xg);
    return hipGetLastError();
}

hipError_t launch_dgf_mix(const float *z, const float *h1, const float *h2, int n, int d, float *x0, hipStream_t s)
{
    if (n < 1 || n > DV_TREE_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_dgf_mix, dim3(n), dim3(PF_THREADS), 0, s, z, h1, h2, d, x0);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const float *src, const RowIndex &ix, int n, int d, float *dst, hipStream_t s)
{
    if (n < 1 || n > DV_TREE_MAX || d % 4) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_gather_rows, dim3(n), dim3(PF_THREADS), 0, s, src, ix, d, dst);
    return hipGetLastError();
}

hipError_t launch_topk_probs(const float *logits, int V, const TopkArgs &a, int n_rows, hipStream_t s)
{
    if (n_rows < 1 || n_rows > DV_TREE_MAX || a.k < 1 || a.k > DV_TOPK_MAX || V > 32 * 1024) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_topk_probs, dim3(n_rows), dim3(1024), 0, s, logits, V, a);
    return hipGetLastError();
}
