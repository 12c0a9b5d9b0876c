// Host side of libdv: argument validation, tree preprocessing, workspace,
// the per-step launch sequence, KV commit and prefill.  Declarations and the
// contract of every entry point are in include/dv.h.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "dv.h"
#include "dv_internal.h"

namespace {

thread_local std::string g_init_error;

struct LayerW {
    const void *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *w_gate, *w_up, *w_down;
    const float *sq = nullptr, *sk = nullptr, *sv = nullptr, *so = nullptr, *sg = nullptr, *su = nullptr,
                *sd = nullptr;  // int8: row scales as passed in
    uint16_t *pk_qkv = nullptr, *pk_o = nullptr, *pk_gu = nullptr, *pk_down = nullptr;
    float *ps_qkv = nullptr, *ps_o = nullptr, *ps_gu = nullptr, *ps_down = nullptr;  // int8: packed-order scales
};

struct GemmPlan {
    int n_tiles = 0;   // 32-row tiles
    int mfma = 0;      // MFMA kernel (bf16 weights, K % 32 == 0) or VALU
    int rb = 0;        // MFMA: 16-row blocks per row group
    int n_groups = 0;  // row groups (VALU: tiles)
    int ks = 1;        // K splits per row group (residual projections)
};

struct ProfEv {
    int cls;
    hipEvent_t a, b;
};

}  // namespace

struct dv_handle {
    dv_config cfg{};
    hipStream_t stream = nullptr;
    int bf16 = 0;          // 16-bit embedding, gains and KV cache; MFMA projections
    int wkind = W_F32;     // projection weights: W_F32, W_BF16 or W_I8
    size_t esz = 4;
    const void *embed = nullptr, *final_norm = nullptr, *lm_head = nullptr;
    std::vector<LayerW> layers;

    // workspace (device)
    float *x = nullptr, *u = nullptr, *q = nullptr, *attn = nullptr, *hbuf = nullptr;
    float *ssq = nullptr;  // per-token partial sums of squares, [64][ssq_max]
    int ssq_max = 0;
    float *part_gemm = nullptr;  // split-K partials of the residual projections
    uint32_t *cnt = nullptr;     // their per-row-group arrival counters
    size_t part_elems = 0;       // floats in part_gemm
    int cnt_n = 0;               // counters in cnt
    uint16_t *u_s = nullptr, *attn_s = nullptr, *h_s = nullptr;  // split-layout activations
    float *part_o = nullptr, *part_m = nullptr, *part_l = nullptr;
    uint32_t *attn_cnt = nullptr;  // per-head arrivals of the attention splits
    int attn_split_max = 0;
    float *arg_val = nullptr;
    int32_t *arg_idx = nullptr;
    float *rope_cos = nullptr, *rope_sin = nullptr;
    uint16_t *pk_lm = nullptr;
    const float *lm_scale = nullptr;
    float *ps_lm = nullptr;
    StepDesc *h_sd = nullptr;  // the step's tree (kernels get it by value)
    DevAccept *d_acc = nullptr, *h_acc = nullptr;
    float *logits_ws = nullptr;  // [max_tree][vocab] logits of a sampled step without out_logits
    // large-M prefill (allocated at its first use, sized for pf_cap tokens,
    // a multiple of 128): residual stream, rotated queries, the split-layout
    // operands (norm numerators, attention output, SwiGLU output) and the
    // norms' sums of squares over 64-row slices
    int pf_cap = 0;
    int32_t *pf_tok = nullptr;
    float *pf_x = nullptr, *pf_q = nullptr, *pf_ssq = nullptr;
    uint16_t *pf_us = nullptr, *pf_as = nullptr, *pf_hs = nullptr;
    // draft side
    bool draft = false;
    const void *dgf_h = nullptr, *dgf_e = nullptr, *dgf_g = nullptr;  // W_h, W_e [d][d], W_g [d][2d]
    GemmPlan p_dgf_d, p_dgf_g;    // projections of W_h / W_e (K = d) and W_g (K = 2 d)
    uint16_t *pk_dh = nullptr, *pk_de = nullptr, *pk_dg = nullptr;  // their MFMA block order
    uint16_t *dgf_xf = nullptr, *dgf_xe = nullptr, *dgf_xg = nullptr;  // split-layout operands
    float *dgf_h1 = nullptr, *dgf_h2 = nullptr, *dgf_z = nullptr;       // [64][d] outputs
    const float *x_in = nullptr;  // stack input rows for the next forward (null: embeddings)
    float *feat_a = nullptr, *feat_b = nullptr;  // [DV_TREE_MAX + 1][d] draft features (row 64: the root's input)
    int32_t *tk_tok = nullptr, *tk_tok_h = nullptr;
    float *tk_p = nullptr, *tk_p_h = nullptr;
    float *p_ws = nullptr;       // [2][vocab] current / residual distribution of the sampling walk
    GemmPlan p_qkv, p_o, p_gu, p_down, p_lm;
    int n_cu = 256;

    // pending (uncommitted) step
    bool pending = false;
    int32_t pend_n = 0, pend_base = 0;
    int32_t pend_parents[DV_TREE_MAX];
    void *pend_k = nullptr, *pend_v = nullptr;

    bool poisoned = false;
    std::string err;

    // per-kernel-class event timing
    int prof = 0;  // class mask
    bool prof_open = false;
    std::vector<hipEvent_t> ev_pool;
    std::vector<ProfEv> ev_live;
    double prof_ms[DV_K_COUNT] = {0, 0, 0, 0};
    int64_t prof_n[DV_K_COUNT] = {0, 0, 0, 0};
};

namespace {

int set_err(dv_handle *h, int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (h) h->err = buf;
    else g_init_error = buf;
    return code;
}

int hip_fail(dv_handle *h, hipError_t e, const char *what)
{
    if (h) h->poisoned = true;
    return set_err(h, DV_EHIP, "HIP error in %s: %s", what, hipGetErrorString(e));
}

#define HIPCHK(h, call)                                        \
    do {                                                       \
        hipError_t e_ = (call);                                \
        if (e_ != hipSuccess) return hip_fail((h), e_, #call); \
    } while (0)

int ceil_div(int a, int b) { return (a + b - 1) / b; }
int round_up(int a, int b) { return ceil_div(a, b) * b; }

// Row groups of 4 blocks (2 where the block count is not a multiple of 4): a
// workgroup then streams 4 KB of weights per 2 KB of shared activations per
// k-step.  Residual projections (d_model rows, too few groups to cover the
// CUs) split K so that groups x splits covers the CUs about once, keeping at
// least 4 k-steps per wave and split; the last split to finish folds them.
GemmPlan make_plan(int n_tiles, int K, int mfma, bool resid, int n_cu)
{
    GemmPlan p;
    p.n_tiles = n_tiles;
    p.mfma = mfma;
    if (mfma) {
        const int blocks = 2 * n_tiles;
        p.rb = blocks % 4 == 0 ? 4 : 2;
        p.n_groups = blocks / p.rb;
        if (resid) {
            const int S = K / 32, nw = gemm_shape(p.rb).nw;
            int ks = std::max(1, (n_cu + p.n_groups / 2) / p.n_groups);
            ks = std::min(ks, std::max(1, S / (4 * nw)));
            p.ks = std::min(ks, 16);
        }
    } else {
        p.n_groups = n_tiles;
    }
    return p;
}

int gemm_units(const GemmPlan &p) { return p.n_groups * p.ks; }

// A projection without K splits whose 4-block groups outnumber the CUs runs
// its steps of at most one token tile as 8-block groups when those fit on the
// CUs once: every CU then streams one group (half the activation bytes per
// weight byte) instead of some CUs streaming two and the rest one.  The
// k-major block order is the same for both group sizes, so the packed weights
// serve either.
GemmPlan step_plan(const GemmPlan &p, int epi, int wkind, int mt, int n_cu)
{
    if (!p.mfma || p.rb != 4 || p.ks != 1 || mt > 1 || p.n_groups % 2) return p;
    if (p.n_groups <= n_cu || p.n_groups / 2 > n_cu || !gemm_has_rb8(epi, wkind, mt)) return p;
    GemmPlan q = p;
    q.rb = 8;
    q.n_groups = p.n_groups / 2;
    return q;
}

// Grid of a launch: every unit its own workgroup, capped at what the CUs hold
// at once (the workgroups then loop over the units).
int gemm_grid(const GemmPlan &p, int epi, int wkind, int mt, int n_cu)
{
    const int cap = std::max(1, gemm_blocks_per_cu(epi, wkind, p.mfma, mt, p.rb) * n_cu);
    return std::min(gemm_units(p), cap);
}

// Event pair for the next launch of class cls, or nullptr when that class is
// not being timed.  GEMM launches pass the pair to hipExtLaunchKernel (the
// dispatch packet records the timestamps); other classes are bracketed by
// hipEventRecord.
ProfEv *prof_pair(dv_handle *h, int cls)
{
    if (!(h->prof >> cls & 1)) return nullptr;
    ProfEv e{cls, nullptr, nullptr};
    if (h->ev_pool.size() >= 2) {
        e.a = h->ev_pool.back(); h->ev_pool.pop_back();
        e.b = h->ev_pool.back(); h->ev_pool.pop_back();
    } else {
        (void)hipEventCreate(&e.a);
        (void)hipEventCreate(&e.b);
    }
    h->ev_live.push_back(e);
    return &h->ev_live.back();
}

void prof_begin(dv_handle *h, int cls)
{
    h->prof_open = false;
    ProfEv *e = prof_pair(h, cls);
    if (!e) return;
    (void)hipEventRecord(e->a, h->stream);
    h->prof_open = true;
}

void prof_end(dv_handle *h)
{
    if (!h->prof_open) return;
    h->prof_open = false;
    (void)hipEventRecord(h->ev_live.back().b, h->stream);
}

// after a stream sync: fold recorded event pairs into the totals
void prof_collect(dv_handle *h)
{
    for (auto &e : h->ev_live) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, e.a, e.b) == hipSuccess) {
            h->prof_ms[e.cls] += ms;
            h->prof_n[e.cls] += 1;
        }
        h->ev_pool.push_back(e.a);
        h->ev_pool.push_back(e.b);
    }
    h->ev_live.clear();
}

int check_tree(dv_handle *h, const int32_t *parents, int n, int base, int32_t *pos,
               int32_t *depth, uint64_t *anc)
{
    int rc = dv_tree_prepare(parents, n, base, pos, depth, anc);
    if (rc != DV_OK) return set_err(h, rc, "invalid draft tree (parents[0] must be -1, 0 <= parents[i] < i, 1 <= n_tree <= 64)");
    return DV_OK;
}

// Enqueue the forward pass over the tree described by h->h_sd (already
// filled) and, when with_head, the lm_head, argmax and acceptance kernels
// (the greedy rule, or the sampling rule when smp is given; out_logits must
// then be non-null, and smp's logits are set to it).
int enqueue_forward(dv_handle *h, const dv_kv *kv, float *out_logits, bool with_head,
                    SampleArgs *smp = nullptr)
{
    const dv_config &c = h->cfg;
    StepDesc *sd = h->h_sd;
    const int M = sd->M, Mpad = sd->Mpad, P = sd->P, half = sd->half;
    const int d = c.d_model, hd = c.head_dim, H = c.n_heads, F = c.d_ffn;
    hipStream_t s = h->stream;
    const int mt = half ? 0 : Mpad / 16;  // token tiles of the split activations (0: half layout)

    const size_t layer_kv = (size_t)H * kv->capacity * hd * h->esz;
    // attention: the P + M keys of each head are split evenly into
    // tile-aligned ranges, one workgroup each, so that heads x splits covers
    // the compute units once (each workgroup streams its range with a
    // two-tile pipeline per wave); the last split of a head to finish merges
    // them (bf16 cache; the fp32 path uses the merge kernel), and a single
    // split writes the output itself
    const int total = P + M;
    int kps, n_split;
    if (h->bf16) {
        n_split = std::max(1, std::min(h->n_cu / H, h->attn_split_max));
        kps = round_up(ceil_div(total, n_split), DV_ATTN_TILE);
    } else {
        kps = round_up(ceil_div(total, h->attn_split_max), DV_ATTN_TILE);
    }
    n_split = ceil_div(total, kps);

    GemmArgs g{};
    g.M = M;
    g.Mpad = Mpad;
    g.half = half;
    g.cap = kv->capacity;
    g.P = P;
    g.hd = hd;
    g.rope_cos = h->rope_cos;
    g.rope_sin = h->rope_sin;
    std::memcpy(g.pos, sd->pos, sizeof g.pos);
    g.eps = c.rms_eps;
    g.dn = d;
    g.resid = h->x;
    g.u = h->u;
    g.us = h->bf16 ? h->u_s : nullptr;  // x * gain feeds QKV, gate/up and lm_head
    g.ssq_out = h->ssq;
    g.part = h->part_gemm;
    g.cnt = h->cnt;
    g.out_split = h->p_down.mfma ? h->h_s : nullptr;  // SWIGLU output feeds the down projection
    g.ssq_in = h->ssq;
    g.n_ssq_in = DV_NORM_SLICES;  // the embedding norm's slices feed the first QKV

    AttnArgs aa{};
    aa.q = h->q;
    aa.cap = kv->capacity;
    aa.hd = hd;
    aa.H = H;
    aa.keys_per_split = kps;
    aa.n_split = n_split;
    aa.tm.M = M;
    aa.tm.P = P;
    aa.tm.Mpad = Mpad;
    aa.tm.half = half;
    std::memcpy(aa.tm.anc, sd->anc, sizeof aa.tm.anc);
    aa.part_o = h->part_o;
    aa.part_m = h->part_m;
    aa.part_l = h->part_l;
    aa.cnt = h->attn_cnt;
    aa.out = h->attn;
    aa.out_split = h->p_o.mfma ? h->attn_s : nullptr;

    auto gemm = [&](const GemmPlan &p0, int epi, const void *w0, const void *w1, const void *w2,
                    const uint16_t *packed, const float *scale, int N, int K, const float *x, const uint16_t *xs,
                    float *out, const void *gain) -> int {
        const GemmPlan p = step_plan(p0, epi, h->wkind, mt, h->n_cu);
        GemmArgs a = g;
        a.packed = packed;
        a.scale = scale;
        a.xs = xs;
        a.w0 = w0;
        a.w1 = w1;
        a.w2 = w2;
        a.N = N;
        a.K = K;
        a.n_tiles = p.n_tiles;
        a.rb = p.rb;
        a.n_groups = p.n_groups;
        a.ks = p.ks;
        a.n_units = gemm_units(p);
        a.x = x;
        a.out = out;
        a.gain = gain;
        const int grid = gemm_grid(p, epi, h->wkind, mt, h->n_cu);
        ProfEv *ev = prof_pair(h, DV_K_GEMM);
        hipError_t e = launch_gemm(a, grid, epi, h->wkind, p.mfma, s, ev ? ev->a : nullptr, ev ? ev->b : nullptr);
        if (e != hipSuccess) return hip_fail(h, e, "gemm launch");
        // the next projection normalises with this one's sums of squares
        if (epi == EPI_RESID) g.n_ssq_in = p.n_groups;
        return DV_OK;
    };

    {
        NormArgs na{};
        na.x = h->x;
        na.embed = h->embed;
        na.gain = h->layers[0].attn_norm;
        na.u = h->u;
        na.us = h->bf16 ? h->u_s : nullptr;
        na.ssq = h->ssq;
        na.d = d;
        na.M = M;
        na.half = half;
        na.x_in = h->x_in;
        std::memcpy(na.tokens, sd->tokens, sizeof na.tokens);
        prof_begin(h, DV_K_NORM);
        hipError_t e = launch_embed_norm(na, Mpad, h->bf16, s);
        prof_end(h);
        if (e != hipSuccess) return hip_fail(h, e, "embedding norm launch");
    }
    int rc;
    for (int l = 0; l < c.n_layers; ++l) {
        const LayerW &w = h->layers[l];
        g.kc = (char *)kv->k + l * layer_kv;
        g.vc = (char *)kv->v + l * layer_kv;
        if ((rc = gemm(h->p_qkv, EPI_QKV, w.wq, w.wk, w.wv, w.pk_qkv, w.ps_qkv, d, d, h->u, h->u_s, h->q, nullptr)))
            return rc;
        aa.kc = g.kc;
        aa.vc = g.vc;
        prof_begin(h, DV_K_ATTN);
        hipError_t e = launch_attention(aa, h->bf16, s);
        // (the bf16 kernel merges its splits itself)
        if (e == hipSuccess && n_split > 1 && !h->bf16) e = launch_attn_merge(aa, Mpad, s);
        prof_end(h);
        if (e != hipSuccess) return hip_fail(h, e, "attention launch");
        if ((rc = gemm(h->p_o, EPI_RESID, w.wo, nullptr, nullptr, w.pk_o, w.ps_o, d, d, h->attn, h->attn_s, nullptr,
                       w.ffn_norm)))
            return rc;
        if ((rc = gemm(h->p_gu, EPI_SWIGLU, w.w_gate, w.w_up, nullptr, w.pk_gu, w.ps_gu, F, d, h->u, h->u_s, h->hbuf,
                       nullptr)))
            return rc;
        const void *next_gain = l + 1 < c.n_layers ? h->layers[l + 1].attn_norm : h->final_norm;
        if ((rc = gemm(h->p_down, EPI_RESID, w.w_down, nullptr, nullptr, w.pk_down, w.ps_down, d, F, h->hbuf, h->h_s,
                       nullptr, next_gain)))
            return rc;
    }
    if (!with_head) return DV_OK;
    g.arg_val = h->arg_val;
    g.arg_idx = h->arg_idx;
    if ((rc = gemm(h->p_lm, EPI_LOGITS, h->lm_head, nullptr, nullptr, h->pk_lm, h->ps_lm, c.vocab, d, h->u, h->u_s,
                   out_logits, nullptr)))
        return rc;
    if (smp) {
        smp->logits = out_logits;
        prof_begin(h, DV_K_OTHER);
        hipError_t e = launch_accept_sampled(*smp, s);
        prof_end(h);
        if (e != hipSuccess) return hip_fail(h, e, "sampled accept launch");
        return DV_OK;
    }
    AcceptArgs ac{};
    ac.arg_val = h->arg_val;
    ac.arg_idx = h->arg_idx;
    ac.n_parts = step_plan(h->p_lm, EPI_LOGITS, h->wkind, mt, h->n_cu).n_groups;  // the lm_head launch's groups
    ac.M = M;
    ac.Mpad = Mpad;
    std::memcpy(ac.tokens, sd->tokens, sizeof ac.tokens);
    std::memcpy(ac.parents, sd->parents, sizeof ac.parents);
    std::memcpy(ac.depth, sd->depth, sizeof ac.depth);
    ac.acc = h->d_acc;
    prof_begin(h, DV_K_OTHER);
    hipError_t e = launch_accept(ac, s);
    prof_end(h);
    if (e != hipSuccess) return hip_fail(h, e, "accept launch");
    return DV_OK;
}

void fill_desc(StepDesc *sd, const int32_t *tokens, const int32_t *parents, int n, int base,
               const int32_t *pos, const int32_t *depth, const uint64_t *anc)
{
    std::memset(sd, 0, sizeof *sd);
    sd->M = n;
    sd->P = base;
    sd->Mpad = round_up(n, 16);
    // up to 8 nodes: hi and lo of the split activations share one MFMA operand
    sd->half = n <= 8 ? 1 : 0;
    for (int i = 0; i < n; ++i) {
        sd->tokens[i] = tokens[i];
        sd->parents[i] = parents[i];
        sd->pos[i] = pos[i];
        sd->depth[i] = depth[i];
        sd->anc[i] = anc[i];
    }
}

// Validate the sampling inputs of a step over an n-node tree and fill the
// walk's arguments (logits are set by the caller).
int prepare_sampled(dv_handle *h, const int32_t *tokens, const int32_t *parents, int n, int vocab,
                    const float *draft_probs, float temperature, const float *u_accept,
                    const float *u_bonus, float *p_ws, DevAccept *acc, SampleArgs *sa)
{
    if (!draft_probs || !u_accept || !u_bonus) return set_err(h, DV_EINVAL, "null draft distribution or uniforms");
    if (reinterpret_cast<uintptr_t>(draft_probs) % 16)
        return set_err(h, DV_EINVAL, "draft_probs must be 16-byte aligned");
    if (!(temperature > 0.f) || !std::isfinite(temperature) || !std::isfinite(1.f / temperature))
        return set_err(h, DV_EINVAL, "temperature must be finite and > 0 (got %g)", (double)temperature);
    for (int i = 0; i < n; ++i) {
        if (!(u_bonus[i] >= 0.f && u_bonus[i] < 1.f))
            return set_err(h, DV_EINVAL, "u_bonus[%d] = %g outside [0, 1)", i, (double)u_bonus[i]);
        if (i > 0 && !(u_accept[i] >= 0.f && u_accept[i] < 1.f))
            return set_err(h, DV_EINVAL, "u_accept[%d] = %g outside [0, 1)", i, (double)u_accept[i]);
    }
    std::memset(sa, 0, sizeof *sa);
    sa->q = draft_probs;
    sa->p = p_ws;
    sa->V = vocab;
    sa->M = n;
    sa->inv_t = 1.f / temperature;
    for (int i = 0; i < n; ++i) {
        sa->tokens[i] = tokens[i];
        sa->parents[i] = parents[i];
        sa->u_accept[i] = i > 0 ? u_accept[i] : 0.f;
        sa->u_bonus[i] = u_bonus[i];
    }
    sa->acc = acc;
    return DV_OK;
}

// Large-M prefill: chunks of up to DV_PF_CHUNK tokens, each one causal pass
// through all layers on the prefill GEMM (k_pf_gemm, fused epilogues) and
// the causal attention kernel; bf16 weights whose projections use the packed
// block order.
constexpr int DV_PF_CHUNK = 1024;

bool pf_supported(const dv_handle *h)
{
    const dv_config &c = h->cfg;
    return h->wkind == W_BF16 && h->p_qkv.mfma && h->p_o.mfma && h->p_gu.mfma && h->p_down.mfma &&
           c.d_model % 64 == 0 && (c.head_dim == 64 || c.head_dim == 128);
}

int pf_reserve(dv_handle *h, int tokens)
{
    const int cap = round_up(std::max(tokens, 1), 128);
    if (h->pf_cap >= cap) return DV_OK;
    const dv_config &c = h->cfg;
    for (void *p : {(void *)h->pf_tok, (void *)h->pf_x, (void *)h->pf_q, (void *)h->pf_ssq, (void *)h->pf_us,
                    (void *)h->pf_as, (void *)h->pf_hs})
        if (p) (void)hipFree(p);
    h->pf_tok = nullptr;
    h->pf_x = h->pf_q = h->pf_ssq = nullptr;
    h->pf_us = h->pf_as = h->pf_hs = nullptr;
    h->pf_cap = 0;
    const size_t Mc = cap, d = c.d_model, F = std::max(c.d_ffn, 1);
    auto dalloc = [&](void **p, size_t bytes) -> bool {
        return hipMalloc(p, bytes) == hipSuccess && hipMemset(*p, 0, bytes) == hipSuccess;
    };
    const bool ok = dalloc((void **)&h->pf_tok, Mc * 4) && dalloc((void **)&h->pf_x, Mc * d * 4) &&
                    dalloc((void **)&h->pf_q, Mc * d * 4) && dalloc((void **)&h->pf_ssq, Mc * (d / 64 + 1) * 4) &&
                    dalloc((void **)&h->pf_us, Mc * d * 4) && dalloc((void **)&h->pf_as, Mc * d * 4) &&
                    dalloc((void **)&h->pf_hs, Mc * F * 4);
    if (!ok) return set_err(h, DV_ENOMEM, "prefill workspace for %d tokens: allocation failed", tokens);
    h->pf_cap = cap;
    return DV_OK;
}

int prefill_large(dv_handle *h, const int32_t *tokens, int n, dv_kv *kv, int32_t *out_next_token)
{
    const dv_config &c = h->cfg;
    const int d = c.d_model, F = c.d_ffn, H = c.n_heads, hd = c.head_dim;
    hipStream_t s = h->stream;
    int rc = pf_reserve(h, std::min(n, DV_PF_CHUNK));
    if (rc) return rc;
    auto ck = [&](hipError_t e, const char *what) -> int { return e == hipSuccess ? DV_OK : hip_fail(h, e, what); };
    const size_t layer_kv = (size_t)H * kv->capacity * hd;
    int done = 0;
    while (done < n) {
        const int M = std::min(DV_PF_CHUNK, n - done), Mp = round_up(M, 128), P0 = kv->len;
        HIPCHK(h, hipMemcpyAsync(h->pf_tok, tokens + done, (size_t)M * 4, hipMemcpyHostToDevice, s));
        prof_begin(h, DV_K_NORM);
        rc = ck(launch_pf_embed(h->pf_tok, h->embed, M, Mp, d, h->layers[0].attn_norm, h->pf_x, h->pf_us, h->pf_ssq,
                                s),
                "prefill embedding");
        prof_end(h);
        if (rc) return rc;
        PfArgs base{};
        base.MT = Mp / 16;
        base.M = M;
        base.P0 = P0;
        base.ssq_in = h->pf_ssq;
        base.nsq_in = d / 64;
        base.eps = c.rms_eps;
        base.d = d;
        base.q = h->pf_q;
        base.cap = kv->capacity;
        base.hd = hd;
        base.rope_cos = h->rope_cos;
        base.rope_sin = h->rope_sin;
        base.hs = h->pf_hs;
        base.x = h->pf_x;
        base.us = h->pf_us;
        base.ssq_out = h->pf_ssq;
        auto gemm = [&](int epi, const uint16_t *packed, int rows, int K, const uint16_t *xs, const void *gain) -> int {
            PfArgs a = base;
            a.packed = packed;
            a.NB = rows / 16;
            a.K = K;
            a.xs = xs;
            a.gain = static_cast<const uint16_t *>(gain);
            prof_begin(h, DV_K_GEMM);
            const hipError_t e = launch_pf_gemm(a, epi, s);
            prof_end(h);
            return ck(e, "prefill GEMM");
        };
        for (int l = 0; l < c.n_layers; ++l) {
            const LayerW &w = h->layers[l];
            base.kc = static_cast<uint16_t *>(kv->k) + (size_t)l * layer_kv;
            base.vc = static_cast<uint16_t *>(kv->v) + (size_t)l * layer_kv;
            if ((rc = gemm(EPI_QKV, w.pk_qkv, 3 * d, d, h->pf_us, nullptr))) return rc;
            prof_begin(h, DV_K_ATTN);
            rc = ck(launch_attn_causal(h->pf_q, base.kc, base.vc, M, P0, H, hd, kv->capacity, Mp / 16, h->pf_as, s),
                    "causal attention");
            prof_end(h);
            if (rc) return rc;
            if ((rc = gemm(EPI_RESID, w.pk_o, d, d, h->pf_as, w.ffn_norm))) return rc;
            if ((rc = gemm(EPI_SWIGLU, w.pk_gu, 2 * F, d, h->pf_us, nullptr))) return rc;
            const void *next_gain = l + 1 < c.n_layers ? h->layers[l + 1].attn_norm : h->final_norm;
            if ((rc = gemm(EPI_RESID, w.pk_down, d, F, h->pf_hs, next_gain))) return rc;
        }
        const bool last = done + M == n;
        if (last) {
            // the next token: final norm, lm_head and argmax of the chunk's last
            // token, on the verify step's kernels (a one-node tree)
            NormArgs na{};
            na.x = h->x;
            na.x_in = h->pf_x + (size_t)(M - 1) * d;
            na.gain = h->final_norm;
            na.u = h->u;
            na.us = h->u_s;
            na.ssq = h->ssq;
            na.d = d;
            na.M = 1;
            na.half = 1;
            prof_begin(h, DV_K_NORM);
            rc = ck(launch_embed_norm(na, 16, 1, s), "prefill final norm");
            prof_end(h);
            if (rc) return rc;
            GemmArgs g{};
            g.packed = h->pk_lm;
            g.N = c.vocab;
            g.K = d;
            g.n_tiles = h->p_lm.n_tiles;
            g.rb = h->p_lm.rb;
            g.n_groups = h->p_lm.n_groups;
            g.ks = h->p_lm.ks;
            g.n_units = gemm_units(h->p_lm);
            g.xs = h->u_s;
            g.M = 1;
            g.Mpad = 16;
            g.half = 1;
            g.ssq_in = h->ssq;
            g.n_ssq_in = DV_NORM_SLICES;
            g.eps = c.rms_eps;
            g.dn = d;
            g.arg_val = h->arg_val;
            g.arg_idx = h->arg_idx;
            ProfEv *ev = prof_pair(h, DV_K_GEMM);
            rc = ck(launch_gemm(g, gemm_grid(h->p_lm, EPI_LOGITS, h->wkind, 0, h->n_cu), EPI_LOGITS, h->wkind, 1, s,
                                ev ? ev->a : nullptr, ev ? ev->b : nullptr),
                    "prefill lm_head");
            if (rc) return rc;
            AcceptArgs ac{};
            ac.arg_val = h->arg_val;
            ac.arg_idx = h->arg_idx;
            ac.n_parts = h->p_lm.n_groups;
            ac.M = 1;
            ac.Mpad = 16;
            ac.parents[0] = -1;
            ac.depth[0] = 1;
            ac.acc = h->d_acc;
            prof_begin(h, DV_K_OTHER);
            rc = ck(launch_accept(ac, s), "prefill argmax");
            prof_end(h);
            if (rc) return rc;
            HIPCHK(h, hipMemcpyAsync(h->h_acc, h->d_acc, sizeof(DevAccept), hipMemcpyDeviceToHost, s));
        }
        HIPCHK(h, hipStreamSynchronize(s));  // also keeps the token upload alive until used
        prof_collect(h);
        kv->len += M;
        done += M;
        if (last && out_next_token) *out_next_token = h->h_acc->argmax[0];
    }
    return DV_OK;
}

// Draft forward over an n-node tree (tree already checked, descriptor not
// yet filled): DGF of (feat_in rows, token embeddings), the block stack with
// those rows as input, logits of every node into out_logits, the residual
// stream after the last block into feat_out.
int draft_forward_impl(dv_handle *h, const int32_t *tokens, const int32_t *parents, int n, dv_kv *kv,
                       const int32_t *pos, const int32_t *depth, const uint64_t *anc, const float *feat_in,
                       float *feat_out, float *out_logits)
{
    const dv_config &c = h->cfg;
    const int d = c.d_model;
    hipStream_t s = h->stream;
    int rc = pf_reserve(h, std::max(n, 1));
    if (rc) return rc;
    // gated fusion on the weight-streaming projections: h1 = W_h f, h2 = W_e e,
    // z = W_g [h1 || h2], x0 = sigmoid(z) h1 + (1 - sigmoid(z)) h2
    const int Mpad = round_up(n, 16);
    auto gemm = [&](const GemmPlan &p, const uint16_t *pk, int K, const uint16_t *xs, float *D) -> int {
        GemmArgs a{};
        a.packed = pk;
        a.xs = xs;
        a.N = d;
        a.K = K;
        a.n_tiles = p.n_tiles;
        a.rb = p.rb;
        a.n_groups = p.n_groups;
        a.ks = p.ks;
        a.n_units = gemm_units(p);
        a.M = n;
        a.Mpad = Mpad;
        a.out = D;
        a.part = h->part_gemm;
        a.cnt = h->cnt;
        const int grid = gemm_grid(p, EPI_PLAIN, W_BF16, Mpad / 16, h->n_cu);
        ProfEv *ev = prof_pair(h, DV_K_GEMM);
        hipError_t e = launch_gemm(a, grid, EPI_PLAIN, W_BF16, 1, s, ev ? ev->a : nullptr, ev ? ev->b : nullptr);
        return e == hipSuccess ? DV_OK : hip_fail(h, e, "DGF projection launch");
    };
    DgfTokens t{};
    for (int i = 0; i < n; ++i) t.tok[i] = tokens[i];
    prof_begin(h, DV_K_OTHER);
    hipError_t e = launch_dgf_in(feat_in, h->embed, t, n, Mpad, d, h->dgf_xf, h->dgf_xe, s);
    prof_end(h);
    if (e != hipSuccess) return hip_fail(h, e, "dgf operands");
    if ((rc = gemm(h->p_dgf_d, h->pk_dh, d, h->dgf_xf, h->dgf_h1)) ||
        (rc = gemm(h->p_dgf_d, h->pk_de, d, h->dgf_xe, h->dgf_h2)))
        return rc;
    prof_begin(h, DV_K_OTHER);
    e = launch_dgf_gate_in(h->dgf_h1, h->dgf_h2, n, Mpad, d, h->dgf_xg, s);
    prof_end(h);
    if (e != hipSuccess) return hip_fail(h, e, "dgf gate input");
    if ((rc = gemm(h->p_dgf_g, h->pk_dg, 2 * d, h->dgf_xg, h->dgf_z))) return rc;
    prof_begin(h, DV_K_OTHER);
    e = launch_dgf_mix(h->dgf_z, h->dgf_h1, h->dgf_h2, n, d, h->pf_x, s);
    prof_end(h);
    if (e != hipSuccess) return hip_fail(h, e, "dgf output");
    fill_desc(h->h_sd, tokens, parents, n, kv->len, pos, depth, anc);
    h->x_in = h->pf_x;
    rc = enqueue_forward(h, kv, out_logits, true);
    h->x_in = nullptr;
    if (rc) return rc;
    HIPCHK(h, hipMemcpyAsync(feat_out, h->x, (size_t)n * d * sizeof(float), hipMemcpyDeviceToDevice, s));
    return DV_OK;
}

int check_kv(dv_handle *h, const dv_kv *kv)
{
    if (!kv || !kv->k || !kv->v) return set_err(h, DV_EINVAL, "null KV cache");
    if (kv->capacity < 32 || kv->capacity % 32 || kv->len < 0 || kv->len > kv->capacity)
        return set_err(h, DV_EINVAL, "bad KV cache capacity/len (%d/%d); capacity must be a positive multiple of 32",
                       kv->len, kv->capacity);
    return DV_OK;
}

}  // namespace

extern "C" {

int dv_tree_prepare(const int32_t *parents, int32_t n, int32_t base_len, int32_t *out_pos,
                    int32_t *out_depth, uint64_t *out_anc)
{
    if (!parents || !out_pos || !out_depth || !out_anc) return DV_EINVAL;
    if (n < 1 || n > DV_MAX_TREE || base_len < 0) return DV_EINVAL;
    if (parents[0] != -1) return DV_EINVAL;
    for (int i = 1; i < n; ++i)
        if (parents[i] < 0 || parents[i] >= i) return DV_EINVAL;
    for (int i = 0; i < n; ++i) {
        const int p = parents[i];
        out_depth[i] = p < 0 ? 1 : out_depth[p] + 1;
        out_anc[i] = (p < 0 ? 0ull : out_anc[p]) | (1ull << i);
        out_pos[i] = base_len + out_depth[i] - 1;
    }
    return DV_OK;
}

int dv_verify_init(const dv_config *cfg, const dv_weights *w, void *stream, dv_handle **out)
{
    if (out) *out = nullptr;
    if (!cfg || !w || !out) return set_err(nullptr, DV_EINVAL, "null argument");
    const dv_config &c = *cfg;
    if (c.n_layers < 1 || c.d_model < 32 || c.n_heads < 1 || c.d_ffn < 16 || c.vocab < 32)
        return set_err(nullptr, DV_EINVAL, "bad model shape");
    if (c.head_dim != 64 && c.head_dim != 128)
        return set_err(nullptr, DV_EINVAL, "head_dim must be 64 or 128");
    if ((long)c.n_heads * c.head_dim != c.d_model)
        return set_err(nullptr, DV_EINVAL, "n_heads * head_dim must equal d_model");
    if (c.d_model > 8192) return set_err(nullptr, DV_EINVAL, "d_model above 8192");
    if (c.d_model % 32 || c.vocab % 32 || c.d_ffn % 16)
        return set_err(nullptr, DV_EINVAL, "d_model and vocab must be multiples of 32, d_ffn of 16");
    if (c.weight_dtype != DV_F32 && c.weight_dtype != DV_BF16 && c.weight_dtype != DV_I8)
        return set_err(nullptr, DV_EINVAL, "weight_dtype must be DV_F32, DV_BF16 or DV_I8");
    if (c.weight_dtype == DV_I8 && (c.d_model % 64 || c.d_ffn % 64))
        return set_err(nullptr, DV_EINVAL, "DV_I8 needs d_model and d_ffn multiples of 64");
    if (c.max_tree < 1 || c.max_tree > DV_MAX_TREE)
        return set_err(nullptr, DV_EINVAL, "max_tree must be in [1, 64]");
    if (c.max_ctx < c.max_tree) return set_err(nullptr, DV_EINVAL, "max_ctx < max_tree");
    if (!(c.rms_eps >= 0.f) || !std::isfinite(c.rms_eps) || !(c.rope_base > 0.f))
        return set_err(nullptr, DV_EINVAL, "bad rms_eps or rope_base");
    if (!w->embed || !w->final_norm || !w->lm_head || !w->attn_norm || !w->wq || !w->wk ||
        !w->wv || !w->wo || !w->ffn_norm || !w->w_gate || !w->w_up || !w->w_down)
        return set_err(nullptr, DV_EINVAL, "null weight pointer table");
    for (int l = 0; l < c.n_layers; ++l)
        if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] ||
            !w->ffn_norm[l] || !w->w_gate[l] || !w->w_up[l] || !w->w_down[l])
            return set_err(nullptr, DV_EINVAL, "null weight pointer in layer %d", l);
    if (c.weight_dtype == DV_I8) {
        if (!w->lm_head_scale || !w->wq_scale || !w->wk_scale || !w->wv_scale || !w->wo_scale ||
            !w->w_gate_scale || !w->w_up_scale || !w->w_down_scale)
            return set_err(nullptr, DV_EINVAL, "null row-scale table (DV_I8)");
        for (int l = 0; l < c.n_layers; ++l)
            if (!w->wq_scale[l] || !w->wk_scale[l] || !w->wv_scale[l] || !w->wo_scale[l] ||
                !w->w_gate_scale[l] || !w->w_up_scale[l] || !w->w_down_scale[l])
                return set_err(nullptr, DV_EINVAL, "null row-scale pointer in layer %d", l);
    }

    // weights may have been written by work still queued on another stream
    if (hipDeviceSynchronize() != hipSuccess)
        return set_err(nullptr, DV_EHIP, "device synchronisation before init failed");
    dv_handle *h = new dv_handle;
    h->cfg = c;
    h->stream = (hipStream_t)stream;
    h->bf16 = c.weight_dtype == DV_BF16 || c.weight_dtype == DV_I8;
    h->wkind = c.weight_dtype == DV_I8 ? W_I8 : (c.weight_dtype == DV_BF16 ? W_BF16 : W_F32);
    h->esz = h->bf16 ? 2 : 4;
    h->embed = w->embed;
    h->final_norm = w->final_norm;
    h->lm_head = w->lm_head;
    if (h->wkind == W_I8) h->lm_scale = w->lm_head_scale;
    h->layers.resize(c.n_layers);
    for (int l = 0; l < c.n_layers; ++l)
    {
        LayerW &lw = h->layers[l];
        lw.attn_norm = w->attn_norm[l];
        lw.wq = w->wq[l];
        lw.wk = w->wk[l];
        lw.wv = w->wv[l];
        lw.wo = w->wo[l];
        lw.ffn_norm = w->ffn_norm[l];
        lw.w_gate = w->w_gate[l];
        lw.w_up = w->w_up[l];
        lw.w_down = w->w_down[l];
        if (h->wkind == W_I8) {
            lw.sq = w->wq_scale[l];
            lw.sk = w->wk_scale[l];
            lw.sv = w->wv_scale[l];
            lw.so = w->wo_scale[l];
            lw.sg = w->w_gate_scale[l];
            lw.su = w->w_up_scale[l];
            lw.sd = w->w_down_scale[l];
        }
    }

    const int d = c.d_model, F = c.d_ffn, H = c.n_heads, hd = c.head_dim, V = c.vocab;
    const int mf = h->bf16;
    {
        int dev = 0, ncu = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
            ncu > 0)
            h->n_cu = ncu;
    }
    const int mf_down = mf && (F % 32 == 0);
    h->p_qkv = make_plan(3 * d / DV_GEMM_TILE, d, mf, false, h->n_cu);
    h->p_o = make_plan(d / DV_GEMM_TILE, d, mf, true, h->n_cu);
    h->p_gu = make_plan(F / 16, d, mf, false, h->n_cu);
    h->p_down = make_plan(d / DV_GEMM_TILE, F, mf_down, true, h->n_cu);
    h->p_lm = make_plan(V / DV_GEMM_TILE, d, mf, false, h->n_cu);

    // split-K partials: units x rb x (64 tokens / 16) x 64 lanes x 4 floats
    size_t part_elems = 16;
    int cnt_n = 1;
    for (const GemmPlan *p : {&h->p_o, &h->p_down})
        if (p->ks > 1) {
            part_elems = std::max(part_elems, (size_t)gemm_units(*p) * p->rb * 4 * 64 * 4);
            cnt_n = std::max(cnt_n, p->n_groups);
        }
    h->ssq_max = std::max({DV_NORM_SLICES, h->p_o.n_groups, h->p_down.n_groups});
    h->part_elems = part_elems;
    h->cnt_n = cnt_n;
    h->attn_split_max = std::max(ceil_div(c.max_ctx, DV_ATTN_SPLIT_KEYS), ceil_div(512, H));
    // the split-K and attention partials are addressed with 32-bit byte offsets
    if ((double)part_elems * 4 >= 2147483648.0) {
        dv_verify_free(h);
        return set_err(nullptr, DV_EINVAL, "model too large for the split-K partial buffer");
    }
    if ((double)H * h->attn_split_max * DV_TREE_MAX * hd * 4 >= 2147483648.0) {
        dv_verify_free(h);
        return set_err(nullptr, DV_EINVAL, "max_ctx too large for the attention split buffers");
    }

    auto dalloc = [&](void **p, size_t bytes) -> bool {
        if (hipMalloc(p, bytes) != hipSuccess) return false;
        return hipMemset(*p, 0, bytes) == hipSuccess;
    };
    const size_t rows = DV_TREE_MAX;
    bool ok = dalloc((void **)&h->x, rows * d * 4) && dalloc((void **)&h->u, rows * d * 4) &&
              dalloc((void **)&h->q, rows * d * 4) && dalloc((void **)&h->attn, rows * d * 4) &&
              dalloc((void **)&h->hbuf, rows * F * 4) &&
              dalloc((void **)&h->ssq, rows * h->ssq_max * 4) &&
              dalloc((void **)&h->cnt, (size_t)cnt_n * 4) &&
              dalloc((void **)&h->u_s, (size_t)d * 2 * rows * 2) &&
              dalloc((void **)&h->attn_s, (size_t)d * 2 * rows * 2) &&
              dalloc((void **)&h->h_s, (size_t)F * 2 * rows * 2) &&
              dalloc((void **)&h->part_o, (size_t)H * h->attn_split_max * rows * hd * 4) &&
              dalloc((void **)&h->part_m, (size_t)H * h->attn_split_max * rows * 4) &&
              dalloc((void **)&h->part_l, (size_t)H * h->attn_split_max * rows * 4) &&
              dalloc((void **)&h->attn_cnt, (size_t)H * 4) &&
              dalloc((void **)&h->part_gemm, part_elems * 4) &&
              hipMemset(h->part_gemm, 0xff, part_elems * 4) == hipSuccess &&  // empty split-K slots
              dalloc((void **)&h->arg_val, (size_t)h->p_lm.n_groups * rows * 4) &&
              dalloc((void **)&h->arg_idx, (size_t)h->p_lm.n_groups * rows * 4) &&
              dalloc((void **)&h->rope_cos, (size_t)c.max_ctx * (hd / 2) * 4) &&
              dalloc((void **)&h->rope_sin, (size_t)c.max_ctx * (hd / 2) * 4) &&
              dalloc((void **)&h->d_acc, sizeof(DevAccept)) &&
              dalloc((void **)&h->logits_ws, (size_t)c.max_tree * c.vocab * 4) &&
              dalloc((void **)&h->p_ws, (size_t)2 * c.vocab * 4);
    h->h_sd = new StepDesc();
    ok = ok && hipHostMalloc((void **)&h->h_acc, sizeof(DevAccept), hipHostMallocDefault) == hipSuccess;
    if (!ok) {
        std::string msg = std::string("workspace allocation failed: ") + hipGetErrorString(hipGetLastError());
        dv_verify_free(h);
        return set_err(nullptr, DV_ENOMEM, "%s", msg.c_str());
    }

    // rotary table: angle pos * base^(-2j/hd) in double, stored fp32
    {
        const int half = hd / 2;
        std::vector<float> cs((size_t)c.max_ctx * half), sn((size_t)c.max_ctx * half);
        for (int j = 0; j < half; ++j) {
            const double theta = std::pow((double)c.rope_base, -2.0 * j / hd);
            for (int p = 0; p < c.max_ctx; ++p) {
                const double ang = (double)p * theta;
                cs[(size_t)p * half + j] = (float)std::cos(ang);
                sn[(size_t)p * half + j] = (float)std::sin(ang);
            }
        }
        if (hipMemcpy(h->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
            hipMemcpy(h->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
            dv_verify_free(h);
            return set_err(nullptr, DV_EHIP, "rope table upload failed");
        }
    }
    // MFMA path: keep the projection matrices in tile order (one extra copy of
    // the projection weights in HBM, written once here)
    if (mf) {
        // int8: the weights keep one byte each and the row scales follow the
        // packed row order
        auto pack = [&](const GemmPlan &p, int epi, const void *w0, const void *w1, const void *w2,
                        const float *s0, const float *s1, const float *s2, int N, int K, uint16_t **dst,
                        float **sdst) -> bool {
            if (!p.mfma) return true;
            const size_t elems = (size_t)p.n_tiles * DV_GEMM_TILE * K;
            if (hipMalloc((void **)dst, elems * (h->wkind == W_I8 ? 1 : 2)) != hipSuccess) return false;
            GemmArgs a{};
            a.w0 = w0;
            a.w1 = w1;
            a.w2 = w2;
            a.s0 = s0;
            a.s1 = s1;
            a.s2 = s2;
            a.N = N;
            a.K = K;
            a.n_tiles = p.n_tiles;
            a.rb = p.rb;
            a.n_groups = p.n_groups;
            a.hd = hd;
            if (launch_pack(a, epi, h->wkind, *dst, nullptr) != hipSuccess) return false;
            if (h->wkind != W_I8) return true;
            if (hipMalloc((void **)sdst, (size_t)p.n_tiles * DV_GEMM_TILE * sizeof(float)) != hipSuccess)
                return false;
            return launch_pack_scales(a, epi, *sdst, nullptr) == hipSuccess;
        };
        bool okp = true;
        for (int l = 0; l < c.n_layers && okp; ++l) {
            LayerW &w = h->layers[l];
            okp = pack(h->p_qkv, EPI_QKV, w.wq, w.wk, w.wv, w.sq, w.sk, w.sv, d, d, &w.pk_qkv, &w.ps_qkv) &&
                  pack(h->p_o, EPI_RESID, w.wo, nullptr, nullptr, w.so, nullptr, nullptr, d, d, &w.pk_o, &w.ps_o) &&
                  pack(h->p_gu, EPI_SWIGLU, w.w_gate, w.w_up, nullptr, w.sg, w.su, nullptr, F, d, &w.pk_gu,
                       &w.ps_gu) &&
                  pack(h->p_down, EPI_RESID, w.w_down, nullptr, nullptr, w.sd, nullptr, nullptr, d, F, &w.pk_down,
                       &w.ps_down);
        }
        okp = okp && pack(h->p_lm, EPI_LOGITS, h->lm_head, nullptr, nullptr, h->lm_scale, nullptr, nullptr, V, d,
                          &h->pk_lm, &h->ps_lm);
        if (!okp) {
            std::string msg = std::string("packed weight allocation failed: ") +
                              hipGetErrorString(hipGetLastError());
            dv_verify_free(h);
            return set_err(nullptr, DV_ENOMEM, "%s", msg.c_str());
        }
    }
    if (hipDeviceSynchronize() != hipSuccess) {
        dv_verify_free(h);
        return set_err(nullptr, DV_EHIP, "device synchronisation after init failed");
    }
    *out = h;
    return DV_OK;
}

static int verify_step_impl(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents, int32_t n_tree,
                            dv_kv *kv, float *out_logits, dv_accept *out_accept, const float *draft_probs,
                            float temperature, const float *u_accept, const float *u_bonus, bool sampled)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (h->poisoned) return DV_EHIP;
    if (!tokens || !tree_parents || !out_accept) return set_err(h, DV_EINVAL, "null argument");
    int rc = check_kv(h, kv);
    if (rc) return rc;
    if (n_tree < 1 || n_tree > h->cfg.max_tree)
        return set_err(h, DV_EINVAL, "n_tree %d outside [1, %d]", n_tree, h->cfg.max_tree);
    for (int i = 0; i < n_tree; ++i)
        if (tokens[i] < 0 || tokens[i] >= h->cfg.vocab)
            return set_err(h, DV_EINVAL, "token id %d at node %d outside [0, %d)", tokens[i], i, h->cfg.vocab);
    int32_t pos[DV_MAX_TREE], depth[DV_MAX_TREE];
    uint64_t anc[DV_MAX_TREE];
    if ((rc = check_tree(h, tree_parents, n_tree, kv->len, pos, depth, anc))) return rc;
    if ((long)kv->len + n_tree > kv->capacity || (long)kv->len + n_tree > h->cfg.max_ctx)
        return set_err(h, DV_ECAPACITY, "len %d + n_tree %d exceeds capacity %d / max_ctx %d",
                       kv->len, n_tree, kv->capacity, h->cfg.max_ctx);
    SampleArgs sa;
    if (sampled) {
        if ((rc = prepare_sampled(h, tokens, tree_parents, n_tree, h->cfg.vocab, draft_probs, temperature, u_accept, u_bonus,
                                  h->p_ws, h->d_acc,
                                  &sa)))
            return rc;
        if (out_logits && reinterpret_cast<uintptr_t>(out_logits) % 16)
            return set_err(h, DV_EINVAL, "out_logits must be 16-byte aligned");
        if (!out_logits) out_logits = h->logits_ws;
    }

    fill_desc(h->h_sd, tokens, tree_parents, n_tree, kv->len, pos, depth, anc);
    if ((rc = enqueue_forward(h, kv, out_logits, true, sampled ? &sa : nullptr))) return rc;
    HIPCHK(h, hipMemcpyAsync(h->h_acc, h->d_acc, sizeof(DevAccept), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    prof_collect(h);

    const DevAccept &a = *h->h_acc;
    std::memset(out_accept, 0, sizeof *out_accept);
    out_accept->accept_len = a.accept_len;
    out_accept->bonus_token = a.bonus;
    out_accept->n_tree = n_tree;
    out_accept->base_len = kv->len;
    for (int i = 0; i < a.accept_len && i < DV_MAX_TREE; ++i) out_accept->path[i] = a.path[i];
    if (!sampled)
        for (int i = 0; i < n_tree; ++i) out_accept->argmax[i] = a.argmax[i];

    h->pending = true;
    h->pend_n = n_tree;
    h->pend_base = kv->len;
    h->pend_k = kv->k;
    h->pend_v = kv->v;
    std::memcpy(h->pend_parents, tree_parents, n_tree * sizeof(int32_t));
    return DV_OK;
}

int dv_verify_step(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents, int32_t n_tree,
                   dv_kv *kv, float *out_logits, dv_accept *out_accept)
{
    return verify_step_impl(h, tokens, tree_parents, n_tree, kv, out_logits, out_accept, nullptr, 0.f, nullptr,
                            nullptr, false);
}

int dv_verify_step_sampled(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents, int32_t n_tree,
                           dv_kv *kv, const float *draft_probs, float temperature, const float *u_accept,
                           const float *u_bonus, float *out_logits, dv_accept *out_accept)
{
    return verify_step_impl(h, tokens, tree_parents, n_tree, kv, out_logits, out_accept, draft_probs,
                            temperature, u_accept, u_bonus, true);
}

int dv_accept_sampled(dv_handle *h, const float *logits, const int32_t *tokens, const int32_t *tree_parents,
                      int32_t n_tree, const float *draft_probs, float temperature, const float *u_accept,
                      const float *u_bonus, dv_accept *out_accept)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (h->poisoned) return DV_EHIP;
    if (!logits || !tokens || !tree_parents || !out_accept) return set_err(h, DV_EINVAL, "null argument");
    if (reinterpret_cast<uintptr_t>(logits) % 16) return set_err(h, DV_EINVAL, "logits must be 16-byte aligned");
    if (n_tree < 1 || n_tree > h->cfg.max_tree)
        return set_err(h, DV_EINVAL, "n_tree %d outside [1, %d]", n_tree, h->cfg.max_tree);
    for (int i = 0; i < n_tree; ++i)
        if (tokens[i] < 0 || tokens[i] >= h->cfg.vocab)
            return set_err(h, DV_EINVAL, "token id %d at node %d outside [0, %d)", tokens[i], i, h->cfg.vocab);
    int32_t pos[DV_MAX_TREE], depth[DV_MAX_TREE];
    uint64_t anc[DV_MAX_TREE];
    int rc = check_tree(h, tree_parents, n_tree, 0, pos, depth, anc);
    if (rc) return rc;
    SampleArgs sa;
    if ((rc = prepare_sampled(h, tokens, tree_parents, n_tree, h->cfg.vocab, draft_probs, temperature, u_accept, u_bonus,
                                  h->p_ws, h->d_acc, &sa)))
        return rc;
    sa.logits = logits;
    prof_begin(h, DV_K_OTHER);
    hipError_t e = launch_accept_sampled(sa, h->stream);
    prof_end(h);
    if (e != hipSuccess) return hip_fail(h, e, "sampled accept launch");
    HIPCHK(h, hipMemcpyAsync(h->h_acc, h->d_acc, sizeof(DevAccept), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    prof_collect(h);
    const DevAccept &a = *h->h_acc;
    std::memset(out_accept, 0, sizeof *out_accept);
    out_accept->accept_len = a.accept_len;
    out_accept->bonus_token = a.bonus;
    out_accept->n_tree = n_tree;
    out_accept->base_len = -1;
    for (int i = 0; i < a.accept_len && i < DV_MAX_TREE; ++i) out_accept->path[i] = a.path[i];
    return DV_OK;
}

int dv_accept_sampled_noalloc(const float *logits, const int32_t *tokens, const int32_t *tree_parents,
                              int32_t n_tree, int32_t vocab, const float *draft_probs, float temperature,
                              const float *u_accept, const float *u_bonus, void *stream, dv_accept *out_accept)
{
    // every check comes before the first HIP call
    if (!logits || !tokens || !tree_parents || !out_accept) return set_err(nullptr, DV_EINVAL, "null argument");
    if (reinterpret_cast<uintptr_t>(logits) % 16) return set_err(nullptr, DV_EINVAL, "logits must be 16-byte aligned");
    if (vocab < 4 || vocab % 4) return set_err(nullptr, DV_EINVAL, "vocab must be a positive multiple of 4 (got %d)", vocab);
    if (vocab > DV_NOALLOC_MAX_VOCAB)
        return set_err(nullptr, DV_EINVAL, "vocab %d exceeds the allocation-free workspace limit of %d", vocab,
                       DV_NOALLOC_MAX_VOCAB);
    if (n_tree < 1 || n_tree > DV_MAX_TREE)
        return set_err(nullptr, DV_EINVAL, "n_tree %d outside [1, %d]", n_tree, DV_MAX_TREE);
    for (int i = 0; i < n_tree; ++i)
        if (tokens[i] < 0 || tokens[i] >= vocab)
            return set_err(nullptr, DV_EINVAL, "token id %d at node %d outside [0, %d)", tokens[i], i, vocab);
    int32_t pos[DV_MAX_TREE], depth[DV_MAX_TREE];
    uint64_t anc[DV_MAX_TREE];
    int rc = check_tree(nullptr, tree_parents, n_tree, 0, pos, depth, anc);
    if (rc) return rc;
    SampleArgs sa;
    if ((rc = prepare_sampled(nullptr, tokens, tree_parents, n_tree, vocab, draft_probs, temperature, u_accept,
                              u_bonus, nullptr, nullptr, &sa)))
        return rc;
    void *ws = nullptr;
    hipError_t e = noalloc_scratch(&ws);
    if (e != hipSuccess) return set_err(nullptr, DV_EHIP, "workspace address: %s", hipGetErrorString(e));
    sa.logits = logits;
    sa.acc = static_cast<DevAccept *>(ws);
    sa.p = reinterpret_cast<float *>(static_cast<char *>(ws) + DV_NOALLOC_ACC_BYTES);
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if ((e = launch_accept_sampled(sa, s)) != hipSuccess)
        return set_err(nullptr, DV_EHIP, "sampled accept launch: %s", hipGetErrorString(e));
    DevAccept a;
    if ((e = hipMemcpyAsync(&a, ws, sizeof a, hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return set_err(nullptr, DV_EHIP, "sampled accept result: %s", hipGetErrorString(e));
    std::memset(out_accept, 0, sizeof *out_accept);
    out_accept->accept_len = a.accept_len;
    out_accept->bonus_token = a.bonus;
    out_accept->n_tree = n_tree;
    out_accept->base_len = -1;
    for (int i = 0; i < a.accept_len && i < DV_MAX_TREE; ++i) out_accept->path[i] = a.path[i];
    return DV_OK;
}

int dv_draft_init(const dv_config *cfg, const dv_weights *w, const dv_dgf_weights *dgf, void *stream,
                  dv_handle **out)
{
    if (!cfg || !w || !dgf || !out) return set_err(nullptr, DV_EINVAL, "null argument");
    if (cfg->weight_dtype != DV_BF16) return set_err(nullptr, DV_EINVAL, "the draft model needs bf16 weights");
    if (!dgf->w_hidden || !dgf->w_embed || !dgf->w_gate) return set_err(nullptr, DV_EINVAL, "null DGF weight");
    if (cfg->d_model % 4) return set_err(nullptr, DV_EINVAL, "d_model must be a multiple of 4");
    dv_handle *h = nullptr;
    int rc = dv_verify_init(cfg, w, stream, &h);
    if (rc) return rc;
    h->draft = true;
    h->dgf_h = dgf->w_hidden;
    h->dgf_e = dgf->w_embed;
    h->dgf_g = dgf->w_gate;
    // the gated fusion's matrices in MFMA block order, split over K like the
    // residual projections (d_model output rows)
    const int d = cfg->d_model;
    h->p_dgf_d = make_plan(d / DV_GEMM_TILE, d, 1, true, h->n_cu);
    h->p_dgf_g = make_plan(d / DV_GEMM_TILE, 2 * d, 1, true, h->n_cu);
    size_t need = h->part_elems;
    int need_cnt = h->cnt_n;
    for (const GemmPlan *p : {&h->p_dgf_d, &h->p_dgf_g})
        if (p->ks > 1) {
            need = std::max(need, (size_t)gemm_units(*p) * p->rb * 4 * 64 * 4);
            need_cnt = std::max(need_cnt, p->n_groups);
        }
    auto zalloc = [](void **p, size_t bytes) -> bool {
        return hipMalloc(p, bytes) == hipSuccess && hipMemset(*p, 0, bytes) == hipSuccess;
    };
    bool okd = true;
    if (need > h->part_elems) {
        (void)hipFree(h->part_gemm);
        h->part_gemm = nullptr;
        okd = zalloc((void **)&h->part_gemm, need * 4) && hipMemset(h->part_gemm, 0xff, need * 4) == hipSuccess;
        h->part_elems = okd ? need : 0;
    }
    if (okd && need_cnt > h->cnt_n) {
        (void)hipFree(h->cnt);
        h->cnt = nullptr;
        okd = zalloc((void **)&h->cnt, (size_t)need_cnt * 4);
        h->cnt_n = okd ? need_cnt : 0;
    }
    auto pack = [&](const GemmPlan &p, const void *w, int K, uint16_t **dst) -> bool {
        if (hipMalloc((void **)dst, (size_t)p.n_tiles * DV_GEMM_TILE * K * 2) != hipSuccess) return false;
        GemmArgs a{};
        a.w0 = w;
        a.N = d;
        a.K = K;
        a.n_tiles = p.n_tiles;
        a.rb = p.rb;
        a.n_groups = p.n_groups;
        return launch_pack(a, EPI_PLAIN, W_BF16, *dst, nullptr) == hipSuccess;
    };
    okd = okd && h->p_dgf_d.mfma && h->p_dgf_g.mfma && pack(h->p_dgf_d, h->dgf_h, d, &h->pk_dh) &&
          pack(h->p_dgf_d, h->dgf_e, d, &h->pk_de) && pack(h->p_dgf_g, h->dgf_g, 2 * d, &h->pk_dg) &&
          zalloc((void **)&h->dgf_xf, (size_t)d * 2 * DV_TREE_MAX * 2) &&
          zalloc((void **)&h->dgf_xe, (size_t)d * 2 * DV_TREE_MAX * 2) &&
          zalloc((void **)&h->dgf_xg, (size_t)2 * d * 2 * DV_TREE_MAX * 2) &&
          zalloc((void **)&h->dgf_h1, (size_t)DV_TREE_MAX * d * 4) &&
          zalloc((void **)&h->dgf_h2, (size_t)DV_TREE_MAX * d * 4) &&
          zalloc((void **)&h->dgf_z, (size_t)DV_TREE_MAX * d * 4) && hipDeviceSynchronize() == hipSuccess;
    if (!okd) {
        dv_verify_free(h);
        return set_err(nullptr, DV_ENOMEM, "draft gated-fusion workspace allocation failed");
    }
    const size_t fb = (size_t)(DV_TREE_MAX + 1) * cfg->d_model * sizeof(float);
    bool ok = hipMalloc((void **)&h->feat_a, fb) == hipSuccess && hipMalloc((void **)&h->feat_b, fb) == hipSuccess &&
              hipMalloc((void **)&h->tk_tok, DV_TREE_MAX * DV_TOPK_MAX * 4) == hipSuccess &&
              hipMalloc((void **)&h->tk_p, DV_TREE_MAX * DV_TOPK_MAX * 4) == hipSuccess &&
              hipHostMalloc((void **)&h->tk_tok_h, DV_TREE_MAX * DV_TOPK_MAX * 4, hipHostMallocDefault) == hipSuccess &&
              hipHostMalloc((void **)&h->tk_p_h, DV_TREE_MAX * DV_TOPK_MAX * 4, hipHostMallocDefault) == hipSuccess;
    if (!ok || pf_reserve(h, DV_TREE_MAX) != DV_OK) {
        dv_verify_free(h);
        return set_err(nullptr, DV_ENOMEM, "draft workspace allocation failed");
    }
    *out = h;
    return DV_OK;
}

int dv_draft_forward(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents, int32_t n_tree, dv_kv *kv,
                     const float *feat_in, float *feat_out, float *out_logits)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (h->poisoned) return DV_EHIP;
    if (!h->draft) return set_err(h, DV_ESTATE, "not a draft handle (dv_draft_init)");
    if (!tokens || !tree_parents || !feat_in || !feat_out || !out_logits) return set_err(h, DV_EINVAL, "null argument");
    for (const void *p : {(const void *)feat_in, (const void *)feat_out, (const void *)out_logits})
        if (reinterpret_cast<uintptr_t>(p) % 16) return set_err(h, DV_EINVAL, "device buffers must be 16-byte aligned");
    int rc = check_kv(h, kv);
    if (rc) return rc;
    if (n_tree < 1 || n_tree > h->cfg.max_tree)
        return set_err(h, DV_EINVAL, "n_tree %d outside [1, %d]", n_tree, h->cfg.max_tree);
    for (int i = 0; i < n_tree; ++i)
        if (tokens[i] < 0 || tokens[i] >= h->cfg.vocab)
            return set_err(h, DV_EINVAL, "token id %d at node %d outside [0, %d)", tokens[i], i, h->cfg.vocab);
    int32_t pos[DV_MAX_TREE], depth[DV_MAX_TREE];
    uint64_t anc[DV_MAX_TREE];
    if ((rc = check_tree(h, tree_parents, n_tree, kv->len, pos, depth, anc))) return rc;
    if ((long)kv->len + n_tree > kv->capacity || (long)kv->len + n_tree > h->cfg.max_ctx)
        return set_err(h, DV_ECAPACITY, "len %d + n_tree %d exceeds capacity %d / max_ctx %d", kv->len, n_tree,
                       kv->capacity, h->cfg.max_ctx);
    if ((rc = draft_forward_impl(h, tokens, tree_parents, n_tree, kv, pos, depth, anc, feat_in, feat_out,
                                 out_logits)))
        return rc;
    HIPCHK(h, hipStreamSynchronize(h->stream));
    prof_collect(h);
    h->pending = false;
    return DV_OK;
}

int dv_draft_tree(dv_handle *h, int32_t root_token, const float *root_feature, dv_kv *kv, int32_t depth,
                  int32_t width, int32_t n_tree, int32_t *out_tokens, int32_t *out_parents, float *out_scores)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (h->poisoned) return DV_EHIP;
    if (!h->draft) return set_err(h, DV_ESTATE, "not a draft handle (dv_draft_init)");
    if (!root_feature || !out_tokens || !out_parents) return set_err(h, DV_EINVAL, "null argument");
    if (reinterpret_cast<uintptr_t>(root_feature) % 16) return set_err(h, DV_EINVAL, "root_feature must be 16-byte aligned");
    int rc = check_kv(h, kv);
    if (rc) return rc;
    const dv_config &c = h->cfg;
    if (root_token < 0 || root_token >= c.vocab) return set_err(h, DV_EINVAL, "root token %d outside [0, %d)", root_token, c.vocab);
    if (depth < 1 || depth > DV_MAX_TREE - 1 || width < 1 || width > DV_TOPK_MAX || n_tree < 1 ||
        n_tree > c.max_tree)
        return set_err(h, DV_EINVAL, "depth %d, width %d or n_tree %d out of range (width <= %d, n_tree <= %d)", depth,
                       width, n_tree, DV_TOPK_MAX, c.max_tree);
    if ((long)kv->len + n_tree > kv->capacity || (long)kv->len + n_tree > c.max_ctx)
        return set_err(h, DV_ECAPACITY, "len %d + n_tree %d exceeds capacity %d / max_ctx %d", kv->len, n_tree,
                       kv->capacity, c.max_ctx);
    const int d = c.d_model;
    hipStream_t s = h->stream;
    struct Node {
        int32_t tok, parent;  // parent: node id
        double score;
    };
    std::vector<Node> nodes{{root_token, -1, 1.0}};
    std::vector<int> tree{0}, frontier{0};  // node ids; tree kept in creation order
    std::vector<int> prev_row(1, -1);       // node id -> row of the last forward (-1: none)
    // feat_a rows: the last forward's output features; row DV_TREE_MAX: the root's input
    HIPCHK(h, hipMemcpyAsync(h->feat_a + (size_t)DV_TREE_MAX * d, root_feature, (size_t)d * sizeof(float),
                             hipMemcpyDeviceToDevice, s));
    auto better = [&](int a, int b) { return nodes[a].score > nodes[b].score || (nodes[a].score == nodes[b].score && a < b); };
    for (int r = 0; r < depth && !frontier.empty(); ++r) {
        std::vector<int> chosen = frontier;
        std::sort(chosen.begin(), chosen.end(), better);
        if ((int)chosen.size() > width) chosen.resize(width);
        // one draft pass over the kept tree
        const int n = (int)tree.size();
        int32_t tok[DV_MAX_TREE], par[DV_MAX_TREE], pos[DV_MAX_TREE], dep[DV_MAX_TREE];
        uint64_t anc[DV_MAX_TREE];
        std::vector<int> row(nodes.size(), -1);
        RowIndex gi{};
        for (int i = 0; i < n; ++i) {
            const Node &nd = nodes[tree[i]];
            row[tree[i]] = i;
            tok[i] = nd.tok;
            par[i] = nd.parent < 0 ? -1 : row[nd.parent];
            gi.idx[i] = nd.parent < 0 ? DV_TREE_MAX : prev_row[nd.parent];
        }
        if ((rc = check_tree(h, par, n, kv->len, pos, dep, anc))) return rc;
        hipError_t e = launch_gather_rows(h->feat_a, gi, n, d, h->feat_b, s);
        if (e != hipSuccess) return hip_fail(h, e, "feature gather");
        // feat_b holds the inputs; the outputs go to feat_a rows [0, n)
        if ((rc = draft_forward_impl(h, tok, par, n, kv, pos, dep, anc, h->feat_b, h->feat_a, h->logits_ws)))
            return rc;
        TopkArgs ta{};
        for (size_t j = 0; j < chosen.size(); ++j) ta.rows[j] = row[chosen[j]];
        ta.k = width;
        ta.out_tok = h->tk_tok;
        ta.out_p = h->tk_p;
        prof_begin(h, DV_K_OTHER);
        e = launch_topk_probs(h->logits_ws, c.vocab, ta, (int)chosen.size(), s);
        prof_end(h);
        if (e != hipSuccess) return hip_fail(h, e, "top-k launch");
        HIPCHK(h, hipMemcpyAsync(h->tk_tok_h, h->tk_tok, chosen.size() * DV_TOPK_MAX * 4, hipMemcpyDeviceToHost, s));
        HIPCHK(h, hipMemcpyAsync(h->tk_p_h, h->tk_p, chosen.size() * DV_TOPK_MAX * 4, hipMemcpyDeviceToHost, s));
        HIPCHK(h, hipStreamSynchronize(s));
        prof_collect(h);
        prev_row = row;
        // children, in the order the chosen nodes were ranked
        std::vector<int> fresh;
        for (size_t j = 0; j < chosen.size(); ++j)
            for (int q = 0; q < width; ++q) {
                nodes.push_back({h->tk_tok_h[j * DV_TOPK_MAX + q], chosen[j],
                                 nodes[chosen[j]].score * (double)h->tk_p_h[j * DV_TOPK_MAX + q]});
                fresh.push_back((int)nodes.size() - 1);
            }
        prev_row.resize(nodes.size(), -1);
        // keep the root and the n_tree - 1 best others (a node outside them
        // can never be selected later: its descendants score no higher)
        std::vector<int> cand(tree.begin() + 1, tree.end());
        cand.insert(cand.end(), fresh.begin(), fresh.end());
        std::sort(cand.begin(), cand.end(), better);
        if ((int)cand.size() > n_tree - 1) cand.resize(n_tree - 1);
        std::sort(cand.begin(), cand.end());
        tree.assign(1, 0);
        tree.insert(tree.end(), cand.begin(), cand.end());
        frontier.clear();
        for (int f : fresh)
            if (std::binary_search(cand.begin(), cand.end(), f)) frontier.push_back(f);
    }
    std::vector<int> row(nodes.size(), -1);
    for (size_t i = 0; i < tree.size(); ++i) row[tree[i]] = (int)i;
    for (size_t i = 0; i < tree.size(); ++i) {
        const Node &nd = nodes[tree[i]];
        out_tokens[i] = nd.tok;
        out_parents[i] = nd.parent < 0 ? -1 : row[nd.parent];
        if (out_scores) out_scores[i] = (float)nd.score;
    }
    for (int i = (int)tree.size(); i < n_tree; ++i) {
        out_tokens[i] = -1;
        out_parents[i] = -1;
        if (out_scores) out_scores[i] = 0.f;
    }
    h->pending = false;
    return (int)tree.size();
}

int dv_kv_commit(dv_handle *h, dv_kv *kv, const dv_accept *acc)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (h->poisoned) return DV_EHIP;
    if (!acc) return set_err(h, DV_EINVAL, "null accept struct");
    int rc = check_kv(h, kv);
    if (rc) return rc;
    if (!h->pending) return set_err(h, DV_ESTATE, "no pending verification step to commit");
    if (acc->n_tree != h->pend_n || acc->base_len != h->pend_base || kv->len != h->pend_base ||
        kv->k != h->pend_k || kv->v != h->pend_v)
        return set_err(h, DV_ESTATE, "accept struct or cache does not match the pending step");
    const int n = acc->accept_len;
    if (n < 1 || n > h->pend_n) return set_err(h, DV_EINVAL, "accept_len %d outside [1, %d]", n, h->pend_n);
    if (acc->path[0] != 0) return set_err(h, DV_EINVAL, "path must start at the root");
    bool identity = true;
    for (int k = 1; k < n; ++k) {
        const int node = acc->path[k];
        if (node <= acc->path[k - 1] || node >= h->pend_n || h->pend_parents[node] != acc->path[k - 1])
            return set_err(h, DV_EINVAL, "path is not a root-to-node chain of the pending tree");
        if (node != k) identity = false;
    }
    if (!identity) {
        CommitArgs ca{};
        ca.kc = kv->k;
        ca.vc = kv->v;
        ca.LH = h->cfg.n_layers * h->cfg.n_heads;
        ca.cap = kv->capacity;
        ca.hd = h->cfg.head_dim;
        ca.P = kv->len;
        ca.n = n;
        for (int k = 0; k < n; ++k) ca.path[k] = acc->path[k];
        hipError_t e = launch_kv_commit(ca, h->bf16, h->stream);
        if (e != hipSuccess) return hip_fail(h, e, "kv commit launch");
    }
    kv->len += n;
    h->pending = false;
    return DV_OK;
}

int dv_prefill(dv_handle *h, const int32_t *tokens, int32_t n, dv_kv *kv, int32_t *out_next_token)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (h->poisoned) return DV_EHIP;
    if (!tokens || n < 1) return set_err(h, DV_EINVAL, "empty prompt");
    int rc = check_kv(h, kv);
    if (rc) return rc;
    for (int i = 0; i < n; ++i)
        if (tokens[i] < 0 || tokens[i] >= h->cfg.vocab)
            return set_err(h, DV_EINVAL, "token id %d at %d outside [0, %d)", tokens[i], i, h->cfg.vocab);
    if ((long)kv->len + n > kv->capacity || (long)kv->len + n > h->cfg.max_ctx)
        return set_err(h, DV_ECAPACITY, "prompt of %d does not fit (len %d, capacity %d, max_ctx %d)",
                       n, kv->len, kv->capacity, h->cfg.max_ctx);
    if (pf_supported(h) && n > h->cfg.max_tree) {
        rc = prefill_large(h, tokens, n, kv, out_next_token);
        h->pending = false;
        return rc;
    }
    const int chunk = h->cfg.max_tree;
    int32_t parents[DV_MAX_TREE], pos[DV_MAX_TREE], depth[DV_MAX_TREE];
    uint64_t anc[DV_MAX_TREE];
    for (int i = 0; i < DV_MAX_TREE; ++i) parents[i] = i - 1;
    int done = 0;
    while (done < n) {
        const int c = std::min(chunk, n - done);
        const bool last = done + c == n;
        if ((rc = check_tree(h, parents, c, kv->len, pos, depth, anc))) return rc;
        fill_desc(h->h_sd, tokens + done, parents, c, kv->len, pos, depth, anc);
        if ((rc = enqueue_forward(h, kv, nullptr, last))) return rc;
        if (last) HIPCHK(h, hipMemcpyAsync(h->h_acc, h->d_acc, sizeof(DevAccept), hipMemcpyDeviceToHost, h->stream));
        HIPCHK(h, hipStreamSynchronize(h->stream));
        prof_collect(h);
        kv->len += c;  // a chain's nodes already sit at slots len + k
        done += c;
        if (last && out_next_token) *out_next_token = h->h_acc->argmax[c - 1];
    }
    h->pending = false;
    return DV_OK;
}

void dv_verify_free(dv_handle *h)
{
    if (!h) return;
    if (h->stream) (void)hipStreamSynchronize(h->stream);
    else (void)hipDeviceSynchronize();
    for (void *p : {(void *)h->x, (void *)h->u, (void *)h->q, (void *)h->attn, (void *)h->hbuf,
                    (void *)h->u_s, (void *)h->attn_s, (void *)h->h_s, (void *)h->ssq,
                    (void *)h->part_o, (void *)h->part_m, (void *)h->part_l, (void *)h->attn_cnt, (void *)h->part_gemm, (void *)h->cnt,
                    (void *)h->arg_val, (void *)h->arg_idx, (void *)h->rope_cos,
                    (void *)h->rope_sin, (void *)h->d_acc, (void *)h->logits_ws, (void *)h->p_ws})
        if (p) (void)hipFree(p);
    for (auto &w : h->layers)
        for (void *p : {(void *)w.pk_qkv, (void *)w.pk_o, (void *)w.pk_gu, (void *)w.pk_down, (void *)w.ps_qkv,
                        (void *)w.ps_o, (void *)w.ps_gu, (void *)w.ps_down})
            if (p) (void)hipFree(p);
    if (h->pk_lm) (void)hipFree(h->pk_lm);
    if (h->ps_lm) (void)hipFree(h->ps_lm);
    for (void *p : {(void *)h->feat_a, (void *)h->feat_b, (void *)h->tk_tok, (void *)h->tk_p, (void *)h->pk_dh,
                    (void *)h->pk_de, (void *)h->pk_dg, (void *)h->dgf_xf, (void *)h->dgf_xe, (void *)h->dgf_xg,
                    (void *)h->dgf_h1, (void *)h->dgf_h2, (void *)h->dgf_z})
        if (p) (void)hipFree(p);
    if (h->tk_tok_h) (void)hipHostFree(h->tk_tok_h);
    if (h->tk_p_h) (void)hipHostFree(h->tk_p_h);
    for (void *p : {(void *)h->pf_tok, (void *)h->pf_x, (void *)h->pf_q, (void *)h->pf_ssq, (void *)h->pf_us,
                    (void *)h->pf_as, (void *)h->pf_hs})
        if (p) (void)hipFree(p);
    delete h->h_sd;
    if (h->h_acc) (void)hipHostFree(h->h_acc);
    for (auto &e : h->ev_live) { (void)hipEventDestroy(e.a); (void)hipEventDestroy(e.b); }
    for (auto e : h->ev_pool) (void)hipEventDestroy(e);
    delete h;
}

const char *dv_last_error(const dv_handle *h)
{
    return h ? h->err.c_str() : g_init_error.c_str();
}

int dv_profile_enable(dv_handle *h, int32_t class_mask)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (class_mask < 0 || class_mask >= (1 << DV_K_COUNT))
        return set_err(h, DV_EINVAL, "bad kernel class mask %d", class_mask);
    h->prof = class_mask;
    return DV_OK;
}

int dv_profile_read(dv_handle *h, int32_t cls, double *total_ms, int64_t *launches, int32_t reset)
{
    if (!h) return set_err(nullptr, DV_EINVAL, "null handle");
    if (cls < 0 || cls >= DV_K_COUNT) return set_err(h, DV_EINVAL, "bad kernel class %d", cls);
    if (total_ms) *total_ms = h->prof_ms[cls];
    if (launches) *launches = h->prof_n[cls];
    if (reset) {
        h->prof_ms[cls] = 0;
        h->prof_n[cls] = 0;
    }
    return DV_OK;
}

}  // extern "C"
