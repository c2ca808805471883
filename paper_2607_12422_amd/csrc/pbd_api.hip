// C ABI of the PEFT-BD speculative-step library: validation, buffer layouts,
// weight packing and the kernel sequence of each pass.  See include/pbd.h.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <string>
#include <vector>

#include "pbd_kernels.h"

using namespace pbd;

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int cdiv(int a, int b) { return (a + b - 1) / b; }

thread_local std::string g_init_error;

// Every size and offset the library uses, derived from a validated config.
struct Layout {
    int L, H, NQ, NKV, HD, F, V, r, D, W, Bmax, max_seq, dtype;
    size_t esz;
    int FK, EPL;
    int Mmax, MTmax, TF, nblk, G, QTmax;
    int kb_qkv, kb_o, kb_gu, kb_d, kb_e;
    int ft_qkv, ft_o, ft_gu, ft_d, ft_e;
    int tiles_qkv, tiles_o, tiles_gu, tiles_d, tiles_e;
    int ks_o, ks_d, nqkv, S_max;
    // packed weights (bytes)
    struct LayerOff {
        size_t qkv, o, gu, d, attn_norm, mlp_norm, q_norm, k_norm, a[7];
    };
    std::vector<LayerOff> lay;
    size_t p_embed, p_final_norm, p_rope, packed_bytes;
    // KV cache
    size_t kv_half, kv_bytes;
    // workspace
    size_t w_x, w_part, w_qkv, w_xa, w_xa_t[3], w_xo, w_xo_t, w_xm, w_xm_t[2], w_xd, w_xd_t, w_xf;
    size_t w_xa_lo, w_xo_lo, w_xm_lo, w_xd_lo, w_xf_lo;
    size_t w_attn_o, w_attn_ml, w_arg_val, w_arg_idx, w_tokens, w_pos0, w_nrows, w_status, ws_bytes;
};

int split_k(int kb) {
    if (kb % 4 == 0) return 4;
    if (kb % 2 == 0) return 2;
    return 1;
}

int validate(const pbd_config* c, std::string& err) {
    if (!c) { err = "config is NULL"; return PBD_ERR_INVALID_ARG; }
    char buf[256];
#define PBD_REQ(cond, code, ...)                                  \
    if (!(cond)) {                                                \
        snprintf(buf, sizeof buf, __VA_ARGS__);                   \
        err = buf;                                                \
        return code;                                              \
    }
    PBD_REQ(c->dtype == PBD_DTYPE_F32 || c->dtype == PBD_DTYPE_BF16, PBD_ERR_INVALID_ARG, "dtype %d unknown", c->dtype);
    PBD_REQ(c->n_layers >= 1 && c->n_layers <= 256, PBD_ERR_SHAPE, "n_layers %d out of range", c->n_layers);
    PBD_REQ(c->hidden >= 64 && c->hidden % 64 == 0 && c->hidden <= MAX_NORM_DIM, PBD_ERR_SHAPE,
            "hidden %d must be a multiple of 64 and <= %d", c->hidden, MAX_NORM_DIM);
    PBD_REQ(c->head_dim == 64 || c->head_dim == 128, PBD_ERR_SHAPE, "head_dim %d must be 64 or 128", c->head_dim);
    PBD_REQ(c->n_kv_heads >= 1 && c->n_q_heads >= c->n_kv_heads && c->n_q_heads % c->n_kv_heads == 0,
            PBD_ERR_SHAPE, "n_q_heads %d must be a multiple of n_kv_heads %d", c->n_q_heads, c->n_kv_heads);
    PBD_REQ(c->n_q_heads * c->head_dim <= MAX_SHRINK_DIM, PBD_ERR_SHAPE, "n_q_heads*head_dim too large");
    PBD_REQ(c->ffn >= 64 && c->ffn % 64 == 0 && c->ffn <= MAX_SHRINK_DIM, PBD_ERR_SHAPE,
            "ffn %d must be a multiple of 64 and <= %d", c->ffn, MAX_SHRINK_DIM);
    PBD_REQ(c->vocab >= 16 && c->vocab % 16 == 0, PBD_ERR_SHAPE, "vocab %d must be a positive multiple of 16", c->vocab);
    PBD_REQ(c->mask_id >= 0 && c->mask_id < c->vocab, PBD_ERR_INVALID_ARG, "mask_id %d outside [0, vocab)", c->mask_id);
    PBD_REQ(c->block >= 1 && c->block <= 32, PBD_ERR_SHAPE, "block %d must lie in [1, 32]", c->block);
    const int W = c->block + 1;
    const int G = c->n_q_heads / c->n_kv_heads;
    PBD_REQ(G * W <= 80, PBD_ERR_SHAPE, "query rows per KV head (%d) exceed 80", G * W);
    PBD_REQ(c->lora_rank >= 0 && c->lora_rank <= 64 && c->lora_rank % 8 == 0, PBD_ERR_SHAPE,
            "lora_rank %d must be a multiple of 8 in [0, 64]", c->lora_rank);
    PBD_REQ(c->lora_rank == 0 || c->lora_alpha > 0.f, PBD_ERR_INVALID_ARG, "lora_alpha must be positive");
    PBD_REQ(c->rms_eps > 0.f && c->rope_theta > 0.f, PBD_ERR_INVALID_ARG, "rms_eps and rope_theta must be positive");
    PBD_REQ(c->max_batch >= 1 && c->max_batch * W <= 4096, PBD_ERR_CAPACITY, "max_batch %d too large", c->max_batch);
    PBD_REQ(c->max_seq > W && c->max_seq <= (1 << 20), PBD_ERR_CAPACITY, "max_seq %d out of range", c->max_seq);
    const int qt = cdiv(G * W, 16);
    PBD_REQ(attn_smem_bytes(c->dtype, c->head_dim, qt) <= 64 * 1024, PBD_ERR_SHAPE, "attention tile does not fit in LDS");
#undef PBD_REQ
    return PBD_OK;
}

void make_layout(const pbd_config* c, Layout& y) {
    y.L = c->n_layers; y.H = c->hidden; y.NQ = c->n_q_heads; y.NKV = c->n_kv_heads; y.HD = c->head_dim;
    y.F = c->ffn; y.V = c->vocab; y.r = c->lora_rank; y.D = c->block; y.W = c->block + 1;
    y.Bmax = c->max_batch; y.max_seq = c->max_seq; y.dtype = c->dtype;
    y.esz = c->dtype == PBD_DTYPE_BF16 ? 2 : 4;
    y.EPL = (int)(16 / y.esz);
    y.FK = 4 * y.EPL;
    y.Mmax = y.Bmax * y.W;
    y.MTmax = cdiv(y.Mmax, 16);
    y.TF = cdiv(y.r, y.FK);
    y.nblk = cdiv(y.max_seq, 16);
    y.G = y.NQ / y.NKV;
    y.QTmax = cdiv(y.G * y.W, 16);
    y.nqkv = (y.NQ + 2 * y.NKV) * y.HD;
    y.kb_qkv = y.H / y.FK; y.kb_o = y.NQ * y.HD / y.FK; y.kb_gu = y.H / y.FK; y.kb_d = y.F / y.FK; y.kb_e = y.H / y.FK;
    y.ft_qkv = y.kb_qkv + y.TF; y.ft_o = y.kb_o + y.TF; y.ft_gu = y.kb_gu + y.TF; y.ft_d = y.kb_d + y.TF; y.ft_e = y.kb_e;
    y.tiles_qkv = y.nqkv / 16; y.tiles_o = y.H / 16; y.tiles_gu = 2 * y.F / 16; y.tiles_d = y.H / 16; y.tiles_e = y.V / 16;
    y.ks_o = split_k(y.kb_o);
    y.ks_d = split_k(y.kb_d);
    y.S_max = std::min(64, cdiv(y.max_seq, 16));

    const size_t FR = 1024;  // bytes per fragment
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
    y.p_embed = take((size_t)y.tiles_e * y.ft_e * FR);
    y.lay.resize(y.L);
    for (int l = 0; l < y.L; ++l) {
        Layout::LayerOff& o = y.lay[l];
        o.qkv = take((size_t)y.tiles_qkv * y.ft_qkv * FR);
        o.o = take((size_t)y.tiles_o * y.ft_o * FR);
        o.gu = take((size_t)y.tiles_gu * y.ft_gu * FR);
        o.d = take((size_t)y.tiles_d * y.ft_d * FR);
        o.attn_norm = take(y.H * y.esz);
        o.mlp_norm = take(y.H * y.esz);
        o.q_norm = take(y.HD * y.esz);
        o.k_norm = take(y.HD * y.esz);
        const int in_f[7] = {y.H, y.H, y.H, y.NQ * y.HD, y.H, y.H, y.F};
        for (int i = 0; i < 7; ++i) o.a[i] = take((size_t)y.r * in_f[i] * y.esz);
    }
    y.p_final_norm = take(y.H * y.esz);
    y.p_rope = take((size_t)y.max_seq * (y.HD / 2) * 8);
    y.packed_bytes = off;

    y.kv_half = (size_t)y.L * y.Bmax * y.NKV * y.nblk * 16 * y.HD * y.esz;
    y.kv_bytes = 2 * y.kv_half;

    off = 0;
    const size_t xfr = (size_t)y.MTmax * FR;    // one k step of an operand
    y.w_x = take((size_t)y.Mmax * y.H * 4);
    y.w_part = take((size_t)std::max(y.ks_o, y.ks_d) * y.Mmax * y.H * 4);
    y.w_qkv = take((size_t)y.Mmax * y.nqkv * 4);
    y.w_xa = take(y.kb_qkv * xfr);
    for (int i = 0; i < 3; ++i) y.w_xa_t[i] = take(std::max(y.TF, 1) * xfr);
    y.w_xo = take(y.kb_o * xfr);
    y.w_xo_t = take(std::max(y.TF, 1) * xfr);
    y.w_xm = take(y.kb_gu * xfr);
    for (int i = 0; i < 2; ++i) y.w_xm_t[i] = take(std::max(y.TF, 1) * xfr);
    y.w_xd = take(y.kb_d * xfr);
    y.w_xd_t = take(std::max(y.TF, 1) * xfr);
    y.w_xf = take(y.kb_e * xfr);
    // residual halves of split (bf16 hi + bf16 lo) operands
    const size_t lo = y.dtype == PBD_DTYPE_BF16 ? 1 : 0;
    y.w_xa_lo = take(lo * y.kb_qkv * xfr);
    y.w_xo_lo = take(lo * y.kb_o * xfr);
    y.w_xm_lo = take(lo * y.kb_gu * xfr);
    y.w_xd_lo = take(lo * y.kb_d * xfr);
    y.w_xf_lo = take(lo * y.kb_e * xfr);
    const size_t nrow_part = (size_t)y.Bmax * y.NQ * y.W * y.S_max;
    y.w_attn_o = take(nrow_part * y.HD * 4);
    y.w_attn_ml = take(nrow_part * 2 * 4);
    y.w_arg_val = take((size_t)y.tiles_e * y.Mmax * 4);
    y.w_arg_idx = take((size_t)y.tiles_e * y.Mmax * 4);
    y.w_tokens = take((size_t)y.Mmax * 4);
    y.w_pos0 = take((size_t)y.Bmax * 4);
    y.w_nrows = take((size_t)y.Bmax * 4);
    y.w_status = take(256);
    y.ws_bytes = off;
}

}  // namespace

// Event-pair timing of kernel classes (profiling aid, off by default).
struct Profiler {
    bool on = false;
    std::vector<hipEvent_t> pool;
    size_t used = 0;
    std::vector<std::pair<int, size_t>> recs;   // (class, index of the begin event)
};

struct pbd_ctx {
    pbd_config cfg;
    Layout ly;
    char* packed;
    char* kv;
    char* ws;
    int kps;
    bool split;          // GEMM activation operands as bf16 hi + bf16 residual
    Profiler prof;
    std::string err;
};

namespace {

int fail(pbd_ctx* c, int code, const std::string& msg) {
    if (c) c->err = msg; else g_init_error = msg;
    return code;
}

int hip_fail(pbd_ctx* c, hipError_t e, const char* what) {
    return fail(c, PBD_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define PBD_HIP(ctx, expr, what)                               \
    do {                                                       \
        hipError_t _e = (expr);                                \
        if (_e != hipSuccess) return hip_fail(ctx, _e, what);  \
    } while (0)

hipError_t prof_mark(pbd_ctx* c, hipStream_t st, int kclass, bool begin) {
    Profiler& p = c->prof;
    if (!p.on) return hipSuccess;
    if (p.used == p.pool.size()) {
        hipEvent_t e;
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return err;
        p.pool.push_back(e);
    }
    if (begin) p.recs.push_back({kclass, p.used});
    return hipEventRecord(p.pool[p.used++], st);
}

// Launch `expr` bracketed by profiling events of class `kc`.
#define PBD_TIMED(ctx, st, kc, expr, what)                                   \
    do {                                                                     \
        PBD_HIP(ctx, prof_mark(ctx, st, kc, true), "profile event");         \
        PBD_HIP(ctx, (expr), what);                                          \
        PBD_HIP(ctx, prof_mark(ctx, st, kc, false), "profile event");        \
    } while (0)

struct PassReq {
    int mode, B;
    const int* seq_len;
    const int* anchor;
    const int* drafts;
    const int* prompt;
    const int* lengths;
    int max_len, chunk_pos;
    bool adapter, causal, write_kv;
    int* out_tokens;
    int* seq_len_out;
    float* logits;
};

int run_pass(pbd_ctx* c, const PassReq& q, hipStream_t st) {
    const Layout& y = c->ly;
    char* ws = c->ws;
    char* pk = c->packed;
    const int dt = y.dtype;
    const int W = y.W, B = q.B, M = B * W, MT = cdiv(M, 16);
    const float scale = y.r > 0 ? c->cfg.lora_alpha / (float)y.r : 0.f;
    const bool lora = q.adapter && y.r > 0;
    const bool split = c->split && dt == PBD_DTYPE_BF16;
    float* x = (float*)(ws + y.w_x);
    float* part = (float*)(ws + y.w_part);
    const size_t part_stride = (size_t)y.Mmax * y.H;
    int* pos0 = (int*)(ws + y.w_pos0);
    int* nrows = (int*)(ws + y.w_nrows);
    int* status = (int*)(ws + y.w_status);

    AssembleArgs as{};
    as.mode = q.mode; as.W = W; as.H = y.H; as.vocab = y.V; as.mask_id = c->cfg.mask_id; as.max_seq = y.max_seq;
    as.chunk_pos = q.chunk_pos; as.max_len = q.max_len;
    as.seq_len = q.seq_len; as.anchor = q.anchor; as.drafts = q.drafts; as.prompt = q.prompt; as.lengths = q.lengths;
    as.tokens = (int*)(ws + y.w_tokens); as.pos0 = pos0; as.nrows = nrows; as.status = status;
    as.embed = pk + y.p_embed; as.x = x;
    PBD_TIMED(c, st, PBD_KCLASS_OTHER, launch_assemble(dt, as, B, st), "assemble");

    const int s_launch = std::min(y.S_max, cdiv(y.max_seq, c->kps));
    for (int l = 0; l < y.L; ++l) {
        const Layout::LayerOff& lo = y.lay[l];
        // attention pre-norm (+ LoRA shrink for q, k, v)
        NormArgs na{};
        na.M = M; na.MT = MT; na.H = y.H; na.eps = c->cfg.rms_eps; na.x = x;
        na.partials = part; na.n_partials = l > 0 ? y.ks_d : 0; na.partial_stride = part_stride;
        na.gain = pk + lo.attn_norm; na.xfrag = ws + y.w_xa; na.xfrag_lo = split ? ws + y.w_xa_lo : nullptr;
        na.n_src = lora ? 3 : 0; na.r = y.r; na.scale = scale;
        for (int i = 0; i < 3; ++i) { na.lora_a[i] = pk + lo.a[i]; na.tail[i] = ws + y.w_xa_t[i]; }
        PBD_TIMED(c, st, PBD_KCLASS_NORM, launch_norm(dt, na, st), "attn norm");

        GemmArgs g{};
        g.w = (const uint4*)(pk + lo.qkv); g.n_tiles = y.tiles_qkv; g.ft = y.ft_qkv; g.kb = y.kb_qkv; g.ks = 1;
        g.tail_frags = lora ? y.TF : 0; g.r = y.r; g.tail_mode = TAIL_BY_TILE;
        g.tile_split0 = y.NQ * y.HD / 16; g.tile_split1 = (y.NQ + y.NKV) * y.HD / 16;
        g.x = (const uint4*)(ws + y.w_xa); g.xlo = split ? (const uint4*)(ws + y.w_xa_lo) : nullptr;
        for (int i = 0; i < 3; ++i) g.xt[i] = (const uint4*)(ws + y.w_xa_t[i]);
        g.M = M; g.MT = MT; g.out = (float*)(ws + y.w_qkv); g.ldo = y.nqkv; g.exclude = -1;
        PBD_TIMED(c, st, PBD_KCLASS_GEMM, launch_gemm(dt, g, EPI_STORE, st), "qkv gemm");

        AttnArgs at{};
        at.layer = l; at.max_batch = y.Bmax; at.n_q = y.NQ; at.n_kv = y.NKV; at.nblk = y.nblk; at.W = W; at.G = y.G;
        at.nqkv = y.nqkv; at.kps = c->kps; at.s_launch = s_launch;
        at.causal = q.causal ? 1 : 0; at.write_kv = q.write_kv ? 1 : 0; at.qk_norm = c->cfg.qk_norm ? 1 : 0;
        at.eps = c->cfg.rms_eps; at.scale_log2 = (float)(1.0 / sqrt((double)y.HD) * 1.4426950408889634);
        at.smem_main = attn_smem_main(dt, y.HD, y.QTmax);
        at.pos0 = pos0; at.nrows = nrows; at.qkv = (const float*)(ws + y.w_qkv);
        at.q_norm = pk + lo.q_norm; at.k_norm = pk + lo.k_norm; at.rope = (const float2*)(pk + y.p_rope);
        at.kcache = c->kv; at.vcache = c->kv + y.kv_half;
        at.part_o = (float*)(ws + y.w_attn_o); at.part_ml = (float*)(ws + y.w_attn_ml);
        PBD_TIMED(c, st, PBD_KCLASS_ATTN, launch_attn(dt, y.HD, y.QTmax, at, B, st), "attention");

        CombineArgs cb{};
        cb.M = M; cb.MT = MT; cb.W = W; cb.n_q = y.NQ; cb.head_dim = y.HD; cb.kps = c->kps; cb.s_launch = s_launch;
        cb.r = lora ? y.r : 0; cb.scale = scale; cb.pos0 = pos0;
        cb.part_o = at.part_o; cb.part_ml = at.part_ml; cb.xfrag = ws + y.w_xo;
        cb.xfrag_lo = split ? ws + y.w_xo_lo : nullptr;
        cb.lora_a = lora ? pk + lo.a[3] : nullptr; cb.tail = ws + y.w_xo_t;
        PBD_TIMED(c, st, PBD_KCLASS_COMBINE, launch_combine(dt, cb, st), "attention combine");

        GemmArgs go{};
        go.w = (const uint4*)(pk + lo.o); go.n_tiles = y.tiles_o; go.ft = y.ft_o; go.kb = y.kb_o; go.ks = y.ks_o;
        go.tail_frags = lora ? y.TF : 0; go.r = y.r; go.tail_mode = TAIL_SINGLE;
        go.x = (const uint4*)(ws + y.w_xo); go.xt[0] = (const uint4*)(ws + y.w_xo_t);
        go.xlo = split ? (const uint4*)(ws + y.w_xo_lo) : nullptr;
        go.M = M; go.MT = MT; go.out = part; go.ldo = y.H; go.partial_stride = part_stride; go.exclude = -1;
        PBD_TIMED(c, st, PBD_KCLASS_GEMM, launch_gemm(dt, go, EPI_PARTIAL, st), "o gemm");

        NormArgs nm{};
        nm.M = M; nm.MT = MT; nm.H = y.H; nm.eps = c->cfg.rms_eps; nm.x = x;
        nm.partials = part; nm.n_partials = y.ks_o; nm.partial_stride = part_stride;
        nm.gain = pk + lo.mlp_norm; nm.xfrag = ws + y.w_xm; nm.xfrag_lo = split ? ws + y.w_xm_lo : nullptr;
        nm.n_src = lora ? 2 : 0; nm.r = y.r; nm.scale = scale;
        nm.lora_a[0] = pk + lo.a[4]; nm.lora_a[1] = pk + lo.a[5];
        nm.tail[0] = ws + y.w_xm_t[0]; nm.tail[1] = ws + y.w_xm_t[1];
        PBD_TIMED(c, st, PBD_KCLASS_NORM, launch_norm(dt, nm, st), "mlp norm");

        GemmArgs gu{};
        gu.w = (const uint4*)(pk + lo.gu); gu.n_tiles = y.tiles_gu; gu.ft = y.ft_gu; gu.kb = y.kb_gu; gu.ks = 1;
        gu.tail_frags = lora ? y.TF : 0; gu.r = y.r; gu.tail_mode = TAIL_BY_ROW_HALF;
        gu.x = (const uint4*)(ws + y.w_xm); gu.xlo = split ? (const uint4*)(ws + y.w_xm_lo) : nullptr;
        gu.out_frag_lo = split ? ws + y.w_xd_lo : nullptr;
        gu.xt[0] = (const uint4*)(ws + y.w_xm_t[0]); gu.xt[1] = (const uint4*)(ws + y.w_xm_t[1]);
        gu.M = M; gu.MT = MT; gu.out_frag = ws + y.w_xd; gu.out_MT = MT; gu.exclude = -1;
        PBD_TIMED(c, st, PBD_KCLASS_GEMM, launch_gemm(dt, gu, EPI_SWIGLU, st), "gate/up gemm");

        if (lora) {
            ShrinkArgs sh{};
            sh.M = M; sh.MT = MT; sh.K = y.F; sh.r = y.r; sh.scale = scale;
            sh.xfrag = ws + y.w_xd; sh.lora_a = pk + lo.a[6]; sh.tail = ws + y.w_xd_t;
            sh.xfrag_lo = split ? ws + y.w_xd_lo : nullptr;
            PBD_TIMED(c, st, PBD_KCLASS_NORM, launch_shrink(dt, sh, st), "down shrink");
        }

        GemmArgs gd{};
        gd.w = (const uint4*)(pk + lo.d); gd.n_tiles = y.tiles_d; gd.ft = y.ft_d; gd.kb = y.kb_d; gd.ks = y.ks_d;
        gd.tail_frags = lora ? y.TF : 0; gd.r = y.r; gd.tail_mode = TAIL_SINGLE;
        gd.x = (const uint4*)(ws + y.w_xd); gd.xt[0] = (const uint4*)(ws + y.w_xd_t);
        gd.xlo = split ? (const uint4*)(ws + y.w_xd_lo) : nullptr;
        gd.M = M; gd.MT = MT; gd.out = part; gd.ldo = y.H; gd.partial_stride = part_stride; gd.exclude = -1;
        PBD_TIMED(c, st, PBD_KCLASS_GEMM, launch_gemm(dt, gd, EPI_PARTIAL, st), "down gemm");
    }

    NormArgs nf{};
    nf.M = M; nf.MT = MT; nf.H = y.H; nf.eps = c->cfg.rms_eps; nf.x = x;
    nf.partials = part; nf.n_partials = y.ks_d; nf.partial_stride = part_stride;
    nf.gain = pk + y.p_final_norm; nf.xfrag = ws + y.w_xf; nf.n_src = 0;
    nf.xfrag_lo = split ? ws + y.w_xf_lo : nullptr;
    PBD_TIMED(c, st, PBD_KCLASS_NORM, launch_norm(dt, nf, st), "final norm");

    GemmArgs ge{};
    ge.w = (const uint4*)(pk + y.p_embed); ge.n_tiles = y.tiles_e; ge.ft = y.ft_e; ge.kb = y.kb_e; ge.ks = 1;
    ge.tail_frags = 0; ge.r = 0; ge.tail_mode = TAIL_SINGLE;
    ge.x = (const uint4*)(ws + y.w_xf); ge.M = M; ge.MT = MT;
    ge.xlo = split ? (const uint4*)(ws + y.w_xf_lo) : nullptr;
    ge.logits = q.logits; ge.ldo = y.V;
    ge.arg_val = (float*)(ws + y.w_arg_val); ge.arg_idx = (int*)(ws + y.w_arg_idx);
    ge.exclude = q.mode == PASS_DRAFT ? c->cfg.mask_id : -1;
    PBD_TIMED(c, st, PBD_KCLASS_LMHEAD, launch_gemm(dt, ge, EPI_ARGMAX, st), "lm head");

    ArgmaxArgs am{};
    am.M = M; am.W = W; am.n_tiles = y.tiles_e; am.mode = q.mode; am.chunk_pos = q.chunk_pos;
    am.arg_val = ge.arg_val; am.arg_idx = ge.arg_idx; am.out = q.out_tokens;
    am.lengths = q.lengths; am.nrows = nrows; am.seq_len_out = q.seq_len_out;
    PBD_TIMED(c, st, PBD_KCLASS_OTHER, launch_argmax(am, st), "argmax");
    return PBD_OK;
}

int check_ctx(const pbd_ctx* c) {
    if (!c) { g_init_error = "context is NULL"; return PBD_ERR_INVALID_ARG; }
    return PBD_OK;
}

int resolve_flags(pbd_ctx* c, uint32_t flags, bool adapter_default, bool causal_default, bool& adapter, bool& causal) {
    const uint32_t known = PBD_PASS_ADAPTER_ON | PBD_PASS_ADAPTER_OFF | PBD_PASS_MASK_BLOCK | PBD_PASS_MASK_CAUSAL;
    if (flags & ~known) return fail(c, PBD_ERR_INVALID_ARG, "unknown pass flag bits");
    if ((flags & PBD_PASS_ADAPTER_ON) && (flags & PBD_PASS_ADAPTER_OFF))
        return fail(c, PBD_ERR_INVALID_ARG, "ADAPTER_ON and ADAPTER_OFF both set");
    if ((flags & PBD_PASS_MASK_BLOCK) && (flags & PBD_PASS_MASK_CAUSAL))
        return fail(c, PBD_ERR_INVALID_ARG, "MASK_BLOCK and MASK_CAUSAL both set");
    adapter = (flags & PBD_PASS_ADAPTER_ON) ? true : (flags & PBD_PASS_ADAPTER_OFF) ? false : adapter_default;
    causal = (flags & PBD_PASS_MASK_CAUSAL) ? true : (flags & PBD_PASS_MASK_BLOCK) ? false : causal_default;
    return PBD_OK;
}

int check_batch(pbd_ctx* c, int32_t batch) {
    if (batch < 1 || batch > c->cfg.max_batch) {
        char buf[128];
        snprintf(buf, sizeof buf, "batch %d outside [1, max_batch=%d]", batch, c->cfg.max_batch);
        return fail(c, batch < 1 ? PBD_ERR_INVALID_ARG : PBD_ERR_CAPACITY, buf);
    }
    return PBD_OK;
}

}  // namespace

extern "C" {

size_t pbd_packed_weight_bytes(const pbd_config* cfg) {
    std::string err;
    if (validate(cfg, err) != PBD_OK) return 0;
    Layout y;
    make_layout(cfg, y);
    return y.packed_bytes;
}

size_t pbd_kv_bytes(const pbd_config* cfg) {
    std::string err;
    if (validate(cfg, err) != PBD_OK) return 0;
    Layout y;
    make_layout(cfg, y);
    return y.kv_bytes;
}

size_t pbd_workspace_bytes(const pbd_config* cfg) {
    std::string err;
    if (validate(cfg, err) != PBD_OK) return 0;
    Layout y;
    make_layout(cfg, y);
    return y.ws_bytes;
}

int pbd_init_weights(const pbd_config* cfg, const pbd_weights* canon, void* packed, size_t packed_bytes,
                     void* kv, size_t kv_bytes, void* ws, size_t ws_bytes, pbd_stream_t stream, pbd_ctx** out) {
    if (!out) return fail(nullptr, PBD_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    std::string err;
    int rc = validate(cfg, err);
    if (rc != PBD_OK) return fail(nullptr, rc, err);
    if (!canon || !canon->embed || !canon->final_norm || !canon->layers)
        return fail(nullptr, PBD_ERR_INVALID_ARG, "weights incomplete");
    if (!packed || !kv || !ws) return fail(nullptr, PBD_ERR_INVALID_ARG, "buffer pointer is NULL");
    Layout y;
    make_layout(cfg, y);
    if (packed_bytes < y.packed_bytes || kv_bytes < y.kv_bytes || ws_bytes < y.ws_bytes)
        return fail(nullptr, PBD_ERR_CAPACITY, "a device buffer is smaller than its *_bytes size");
    for (int l = 0; l < y.L; ++l) {
        const pbd_layer_weights& lw = canon->layers[l];
        const void* req[] = {lw.attn_norm, lw.q, lw.k, lw.v, lw.o, lw.mlp_norm, lw.gate, lw.up, lw.down};
        for (const void* p : req)
            if (!p) return fail(nullptr, PBD_ERR_INVALID_ARG, "layer weight pointer is NULL");
        if (cfg->qk_norm && (!lw.q_norm || !lw.k_norm)) return fail(nullptr, PBD_ERR_INVALID_ARG, "qk_norm gains missing");
        if (y.r > 0)
            for (int i = 0; i < 7; ++i)
                if (!lw.lora_a[i] || !lw.lora_b[i]) return fail(nullptr, PBD_ERR_INVALID_ARG, "LoRA pointer is NULL");
    }
    pbd_ctx* c = new (std::nothrow) pbd_ctx();
    if (!c) return fail(nullptr, PBD_ERR_CAPACITY, "out of host memory");
    c->cfg = *cfg;
    c->ly = y;
    c->packed = (char*)packed;
    c->kv = (char*)kv;
    c->ws = (char*)ws;
    c->kps = 128;
    c->split = cfg->dtype == PBD_DTYPE_BF16;
    hipStream_t st = (hipStream_t)stream;
    const int dt = y.dtype;

    auto cleanup_fail = [&](hipError_t e, const char* what) {
        std::string m = std::string(what) + ": " + hipGetErrorString(e);
        delete c;
        return fail(nullptr, PBD_ERR_HIP, m);
    };
#define PBD_INIT_HIP(expr, what)                          \
    do {                                                  \
        hipError_t _e = (expr);                           \
        if (_e != hipSuccess) return cleanup_fail(_e, what); \
    } while (0)

    // zero the workspace (operand padding must be finite) and the cache
    PBD_INIT_HIP(launch_fill_u32(ws, y.ws_bytes / 4, 0u, st), "clear workspace");
    PBD_INIT_HIP(launch_fill_u32(kv, y.kv_bytes / 4, 0u, st), "clear kv");

    auto pack = [&](size_t off, int tiles, int ft, int kb, int K, int map, int n_src, const int* rows,
                    const void* const* w, const void* const* b) {
        PackArgs p{};
        p.n_tiles = tiles; p.ft = ft; p.kb = kb; p.K = K; p.r = y.r; p.row_map = map; p.n_src = n_src;
        for (int i = 0; i < n_src; ++i) { p.src_rows[i] = rows[i]; p.w[i] = w[i]; p.b[i] = b ? b[i] : nullptr; }
        p.dst = c->packed + off;
        return launch_pack(dt, p, st);
    };
    {
        const int rows[1] = {y.V};
        const void* w[1] = {canon->embed};
        PBD_INIT_HIP(pack(y.p_embed, y.tiles_e, y.ft_e, y.kb_e, y.H, MAP_CONCAT, 1, rows, w, nullptr), "pack embed");
    }
    for (int l = 0; l < y.L; ++l) {
        const pbd_layer_weights& lw = canon->layers[l];
        const Layout::LayerOff& lo = y.lay[l];
        const void* const* B = y.r > 0 ? lw.lora_b : nullptr;
        {
            const int rows[3] = {y.NQ * y.HD, y.NKV * y.HD, y.NKV * y.HD};
            const void* w[3] = {lw.q, lw.k, lw.v};
            const void* b[3] = {B ? B[0] : nullptr, B ? B[1] : nullptr, B ? B[2] : nullptr};
            PBD_INIT_HIP(pack(lo.qkv, y.tiles_qkv, y.ft_qkv, y.kb_qkv, y.H, MAP_CONCAT, 3, rows, w, b), "pack qkv");
        }
        {
            const int rows[1] = {y.H};
            const void* w[1] = {lw.o};
            const void* b[1] = {B ? B[3] : nullptr};
            PBD_INIT_HIP(pack(lo.o, y.tiles_o, y.ft_o, y.kb_o, y.NQ * y.HD, MAP_CONCAT, 1, rows, w, b), "pack o");
        }
        {
            const int rows[2] = {y.F, y.F};
            const void* w[2] = {lw.gate, lw.up};
            const void* b[2] = {B ? B[4] : nullptr, B ? B[5] : nullptr};
            PBD_INIT_HIP(pack(lo.gu, y.tiles_gu, y.ft_gu, y.kb_gu, y.H, MAP_INTERLEAVE2, 2, rows, w, b), "pack gate/up");
        }
        {
            const int rows[1] = {y.H};
            const void* w[1] = {lw.down};
            const void* b[1] = {B ? B[6] : nullptr};
            PBD_INIT_HIP(pack(lo.d, y.tiles_d, y.ft_d, y.kb_d, y.F, MAP_CONCAT, 1, rows, w, b), "pack down");
        }
        PBD_INIT_HIP(hipMemcpyAsync(c->packed + lo.attn_norm, lw.attn_norm, y.H * y.esz, hipMemcpyDeviceToDevice, st), "copy norm");
        PBD_INIT_HIP(hipMemcpyAsync(c->packed + lo.mlp_norm, lw.mlp_norm, y.H * y.esz, hipMemcpyDeviceToDevice, st), "copy norm");
        if (cfg->qk_norm) {
            PBD_INIT_HIP(hipMemcpyAsync(c->packed + lo.q_norm, lw.q_norm, y.HD * y.esz, hipMemcpyDeviceToDevice, st), "copy qnorm");
            PBD_INIT_HIP(hipMemcpyAsync(c->packed + lo.k_norm, lw.k_norm, y.HD * y.esz, hipMemcpyDeviceToDevice, st), "copy knorm");
        }
        const int in_f[7] = {y.H, y.H, y.H, y.NQ * y.HD, y.H, y.H, y.F};
        for (int i = 0; i < 7 && y.r > 0; ++i)
            PBD_INIT_HIP(hipMemcpyAsync(c->packed + lo.a[i], lw.lora_a[i], (size_t)y.r * in_f[i] * y.esz,
                                        hipMemcpyDeviceToDevice, st), "copy lora A");
    }
    PBD_INIT_HIP(hipMemcpyAsync(c->packed + y.p_final_norm, canon->final_norm, y.H * y.esz, hipMemcpyDeviceToDevice, st),
                 "copy final norm");
    // RoPE table: angle(pos, i) = pos * theta^(-2i/d), computed in double.
    {
        const int half = y.HD / 2;
        std::vector<float> tab((size_t)y.max_seq * half * 2);
        for (int p = 0; p < y.max_seq; ++p)
            for (int i = 0; i < half; ++i) {
                const double ang = (double)p * pow((double)cfg->rope_theta, -2.0 * i / (double)y.HD);
                tab[((size_t)p * half + i) * 2 + 0] = (float)cos(ang);
                tab[((size_t)p * half + i) * 2 + 1] = (float)sin(ang);
            }
        PBD_INIT_HIP(hipMemcpyAsync(c->packed + y.p_rope, tab.data(), tab.size() * 4, hipMemcpyHostToDevice, st), "rope table");
        PBD_INIT_HIP(hipStreamSynchronize(st), "init sync");
    }
#undef PBD_INIT_HIP
    *out = c;
    return PBD_OK;
}

int pbd_prefill(pbd_ctx* c, int32_t batch, const int32_t* tokens, const int32_t* lengths, int32_t max_len,
                int32_t* seq_len, int32_t* anchor, pbd_stream_t stream) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if ((rc = check_batch(c, batch))) return rc;
    if (!tokens || !lengths || !seq_len || !anchor) return fail(c, PBD_ERR_INVALID_ARG, "NULL pointer argument");
    if (max_len < 1) return fail(c, PBD_ERR_INVALID_ARG, "max_len must be >= 1");
    if (max_len + c->ly.W > c->cfg.max_seq) return fail(c, PBD_ERR_CAPACITY, "max_len + D + 1 exceeds max_seq");
    const int W = c->ly.W;
    for (int cp = 0; cp < max_len; cp += W) {
        PassReq q{};
        q.mode = PASS_PREFILL; q.B = batch; q.prompt = tokens; q.lengths = lengths; q.max_len = max_len;
        q.chunk_pos = cp; q.adapter = false; q.causal = true; q.write_kv = true;
        q.out_tokens = anchor; q.seq_len_out = seq_len;
        if ((rc = run_pass(c, q, (hipStream_t)stream))) return rc;
    }
    return PBD_OK;
}

int pbd_draft_block(pbd_ctx* c, int32_t batch, const int32_t* seq_len, const int32_t* anchor, uint32_t flags,
                    int32_t* draft, float* logits, pbd_stream_t stream) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if ((rc = check_batch(c, batch))) return rc;
    if (!seq_len || !anchor || !draft) return fail(c, PBD_ERR_INVALID_ARG, "NULL pointer argument");
    bool adapter, causal;
    if ((rc = resolve_flags(c, flags, true, false, adapter, causal))) return rc;
    PassReq q{};
    q.mode = PASS_DRAFT; q.B = batch; q.seq_len = seq_len; q.anchor = anchor;
    q.adapter = adapter; q.causal = causal; q.write_kv = false; q.out_tokens = draft; q.logits = logits;
    return run_pass(c, q, (hipStream_t)stream);
}

int pbd_verify_block(pbd_ctx* c, int32_t batch, const int32_t* seq_len, const int32_t* anchor, const int32_t* draft,
                     uint32_t flags, int32_t* verify, float* logits, pbd_stream_t stream) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if ((rc = check_batch(c, batch))) return rc;
    if (!seq_len || !anchor || !draft || !verify) return fail(c, PBD_ERR_INVALID_ARG, "NULL pointer argument");
    bool adapter, causal;
    if ((rc = resolve_flags(c, flags, false, true, adapter, causal))) return rc;
    PassReq q{};
    q.mode = PASS_VERIFY; q.B = batch; q.seq_len = seq_len; q.anchor = anchor; q.drafts = draft;
    q.adapter = adapter; q.causal = causal; q.write_kv = true; q.out_tokens = verify; q.logits = logits;
    return run_pass(c, q, (hipStream_t)stream);
}

int pbd_accept_commit(pbd_ctx* c, int32_t batch, const int32_t* draft, const int32_t* verify, const int32_t* forced_n,
                      int32_t* seq_len, int32_t* anchor, int32_t* n_accepted, int32_t* out_tokens, pbd_stream_t stream) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if ((rc = check_batch(c, batch))) return rc;
    if (!draft || !verify || !seq_len || !anchor || !n_accepted || !out_tokens)
        return fail(c, PBD_ERR_INVALID_ARG, "NULL pointer argument");
    AcceptArgs a{};
    a.B = batch; a.D = c->ly.D; a.max_seq = c->cfg.max_seq;
    a.draft = draft; a.verify = verify; a.forced = forced_n; a.seq_len = seq_len; a.anchor = anchor;
    a.n_acc = n_accepted; a.out = out_tokens; a.status = (int*)(c->ws + c->ly.w_status);
    PBD_HIP(c, launch_accept(a, (hipStream_t)stream), "accept");
    return PBD_OK;
}

int pbd_sync_status(pbd_ctx* c, pbd_stream_t stream, int32_t* status) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if (!status) return fail(c, PBD_ERR_INVALID_ARG, "status is NULL");
    hipStream_t st = (hipStream_t)stream;
    int32_t host = 0;
    void* dev = c->ws + c->ly.w_status;
    PBD_HIP(c, hipMemcpyAsync(&host, dev, sizeof(int32_t), hipMemcpyDeviceToHost, st), "read status");
    PBD_HIP(c, hipStreamSynchronize(st), "sync");
    if (host != 0) {
        PBD_HIP(c, launch_fill_u32(dev, 1, 0u, st), "clear status");
        PBD_HIP(c, hipStreamSynchronize(st), "sync");
    }
    *status = host;
    return PBD_OK;
}

int pbd_set_attn_keys_per_split(pbd_ctx* c, int32_t keys) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if (keys < 16 || keys % 16 != 0) return fail(c, PBD_ERR_INVALID_ARG, "keys per split must be a positive multiple of 16");
    c->kps = keys;
    return PBD_OK;
}

int pbd_set_operand_precision(pbd_ctx* c, int32_t mode) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if (mode != PBD_OPERANDS_BF16 && mode != PBD_OPERANDS_BF16X2)
        return fail(c, PBD_ERR_INVALID_ARG, "unknown operand precision mode");
    c->split = mode == PBD_OPERANDS_BF16X2;
    return PBD_OK;
}

int pbd_profile_enable(pbd_ctx* c, int32_t on) {
    int rc = check_ctx(c);
    if (rc) return rc;
    c->prof.on = on != 0;
    c->prof.used = 0;
    c->prof.recs.clear();
    return PBD_OK;
}

int pbd_profile_read(pbd_ctx* c, int32_t kclass, double* total_ms, int64_t* launches) {
    int rc = check_ctx(c);
    if (rc) return rc;
    if (!total_ms || !launches || kclass < 0 || kclass >= PBD_KCLASS_COUNT)
        return fail(c, PBD_ERR_INVALID_ARG, "bad profile query");
    Profiler& p = c->prof;
    double tot = 0.0;
    int64_t n = 0;
    if (p.used > 0) PBD_HIP(c, hipEventSynchronize(p.pool[p.used - 1]), "profile sync");
    for (const auto& r : p.recs) {
        if (r.first != kclass) continue;
        float ms = 0.f;
        PBD_HIP(c, hipEventElapsedTime(&ms, p.pool[r.second], p.pool[r.second + 1]), "profile elapsed");
        tot += ms;
        ++n;
    }
    *total_ms = tot;
    *launches = n;
    return PBD_OK;
}

const char* pbd_last_error(const pbd_ctx* c) { return c ? c->err.c_str() : g_init_error.c_str(); }

void pbd_destroy(pbd_ctx* c) {
    if (!c) return;
    for (hipEvent_t e : c->prof.pool) (void)hipEventDestroy(e);
    delete c;
}

}  // extern "C"
