// HIP kernels of the PEFT-BD speculative step for gfx950.
//
// One pass (draft or verify, Sec. 3 steps 1-3) runs, per layer:
//   k_norm      fold split-K partials into the fp32 residual, RMSNorm, write the
//               GEMM operand; draft: LoRA shrink u = s * A x (App. A.2)
//   k_gemm      weight-streaming skinny GEMM on MFMA, W x (+ B u when the
//               adapter is on) with a fused epilogue
//   k_attn      split-KV attention partials on MFMA over the committed prefix
//               and the block (bidirectional or causal block mask); QK-norm and
//               RoPE of the block rows; the verify appends the block K/V
//   k_combine   merge the split partials, write the O-projection operand;
//               draft: LoRA shrink of the attention output
// then the final norm, the tied LM head with a fused argmax, and the
// longest-prefix acceptance (Sec. 3 step 4, App. A.1).
#include "pbd_device.h"
#include "pbd_kernels.h"

namespace pbd {

static __device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Split-KV schedule shared by k_attn and k_combine.
static __device__ __forceinline__ void attn_splits(int t, int kps, int s_launch, int& s_eff, int& chunk) {
    s_eff = min(max(ceil_div(t, kps), 1), s_launch);
    chunk = ceil_div(ceil_div(max(t, 1), s_eff), 16) * 16;
}

// ---------------------------------------------------------------------------
// Block assembly and embedding gather (Sec. 3 steps 1 and 3)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_assemble(AssembleArgs a) {
    const int b = blockIdx.x;
    const int W = a.W;
    __shared__ int s_tok[64];
    __shared__ int s_pos, s_nrows;
    if (threadIdx.x == 0) {
        int pos0 = 0, nrows = W;
        bool ok = true;
        if (a.mode == PASS_PREFILL) {
            int len = a.lengths[b];
            if (len < 1 || len > a.max_len || len + W > a.max_seq) ok = false;
            pos0 = a.chunk_pos;
            nrows = ok ? min(max(len - a.chunk_pos, 0), W) : 0;
        } else {
            pos0 = a.seq_len[b];
            if (pos0 < 0 || pos0 + W > a.max_seq) ok = false;
            nrows = ok ? W : 0;
        }
        if (!ok) {
            atomicOr(a.status, PBD_STATUS_CAPACITY);
            pos0 = 0;
        }
        s_pos = pos0;
        s_nrows = nrows;
        a.pos0[b] = pos0;
        a.nrows[b] = nrows;
    }
    __syncthreads();
    if (threadIdx.x < W) {
        const int j = threadIdx.x;
        int tok;
        if (a.mode == PASS_PREFILL) {
            tok = (j < s_nrows) ? a.prompt[(size_t)b * a.max_len + a.chunk_pos + j] : 0;
        } else if (j == 0) {
            tok = a.anchor[b];
        } else if (a.mode == PASS_DRAFT) {
            tok = a.mask_id;
        } else {
            tok = a.drafts[b * (W - 1) + j - 1];
        }
        if (tok < 0 || tok >= a.vocab) {
            if (j < s_nrows) atomicOr(a.status, PBD_STATUS_TOKEN);
            tok = 0;
        }
        s_tok[j] = tok;
        a.tokens[b * W + j] = tok;
    }
    __syncthreads();
    // Gather embedding rows from the fragment-packed table into the fp32 residual.
    const T* E = (const T*)a.embed;
    const int FK = Elt<T>::FK;
    const int ft = a.H / FK;
    for (int idx = threadIdx.x; idx < W * a.H; idx += blockDim.x) {
        int j = idx / a.H, k = idx % a.H;
        int v = s_tok[j];
        size_t off = frag_elem<T>((size_t)(v / 16) * ft + k / FK, v % 16, k % FK);
        a.x[(size_t)(b * W + j) * a.H + k] = to_f32(E[off]);
    }
}

// ---------------------------------------------------------------------------
// RMSNorm with residual fold and LoRA shrink
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_norm(NormArgs a) {
    const int m = blockIdx.x;
    const int H = a.H;
    __shared__ float s_x[MAX_NORM_DIM];
    __shared__ float s_red[8];
    float* xr = a.x + (size_t)m * H;
    float ss = 0.f;
    for (int k = threadIdx.x; k < H; k += blockDim.x) {
        float v = xr[k];
        for (int p = 0; p < a.n_partials; ++p)            // fixed order: deterministic
            v += a.partials[(size_t)p * a.partial_stride + (size_t)m * H + k];
        if (a.n_partials > 0) xr[k] = v;
        s_x[k] = v;
        ss += v * v;
    }
    ss = wave_sum(ss);
    const int wid = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    if (lane == 0) s_red[wid] = ss;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int w = 0; w < (int)(blockDim.x / WAVE); ++w) t += s_red[w];
        s_red[4] = rsqrtf(t / (float)H + a.eps);
    }
    __syncthreads();
    const float inv = s_red[4];
    const T* g = (const T*)a.gain;
    T* xf = (T*)a.xfrag;
    T* xl = (T*)a.xfrag_lo;
    for (int k = threadIdx.x; k < H; k += blockDim.x) {
        const float v = s_x[k] * inv * to_f32(g[k]);
        const T q = from_f32<T>(v);
        const size_t e = xfrag_elem<T>(m, k, a.MT);
        xf[e] = q;
        if (xl) xl[e] = from_f32<T>(v - to_f32(q));
        s_x[k] = xl ? v : to_f32(q);                       // what the GEMM sees
    }
    if (a.n_src == 0) return;
    __syncthreads();
    // u_s[j] = scale * sum_k A_s[j][k] * xn[k], one wave per (source, j).
    const int total = a.n_src * a.r;
    for (int job = wid; job < total; job += blockDim.x / WAVE) {
        int src = job / a.r, j = job % a.r;
        const T* A = (const T*)a.lora_a[src] + (size_t)j * H;
        float acc = 0.f;
        for (int k = lane; k < H; k += WAVE) acc += to_f32(A[k]) * s_x[k];
        acc = wave_sum(acc);
        if (lane == 0) ((T*)a.tail[src])[xfrag_elem<T>(m, j, a.MT)] = from_f32<T>(acc * a.scale);
    }
}

// LoRA shrink of an operand already in fragment layout (the down projection's
// input h): u[m][j] = scale * sum_k A[j][k] h[m][k].
template <typename T>
__global__ __launch_bounds__(256) void k_shrink(ShrinkArgs a) {
    const int m = blockIdx.x;
    __shared__ float s_h[MAX_SHRINK_DIM];
    const T* X = (const T*)a.xfrag;
    const T* XL = (const T*)a.xfrag_lo;
    for (int k = threadIdx.x; k < a.K; k += blockDim.x) {
        const size_t e = xfrag_elem<T>(m, k, a.MT);
        s_h[k] = to_f32(X[e]) + (XL ? to_f32(XL[e]) : 0.f);
    }
    __syncthreads();
    const int wid = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    for (int j = wid; j < a.r; j += blockDim.x / WAVE) {
        const T* A = (const T*)a.lora_a + (size_t)j * a.K;
        float acc = 0.f;
        for (int k = lane; k < a.K; k += WAVE) acc += to_f32(A[k]) * s_h[k];
        acc = wave_sum(acc);
        if (lane == 0) ((T*)a.tail)[xfrag_elem<T>(m, j, a.MT)] = from_f32<T>(acc * a.scale);
    }
}

// ---------------------------------------------------------------------------
// Skinny weight-streaming GEMM:  Y[m][n] = sum_k W[n][k] X[m][k]  (+ LoRA tail)
//
// A work-group owns one 16-row tile of W (and one K split); its four waves take
// the tile's fragments round-robin, so every fragment of W is read once, as one
// contiguous 1 KiB wavefront load, and feeds MG m-tiles of MFMA.  The LoRA
// expand B (A x) is the same contraction over r extra k columns: the packed tile
// carries B's rows after W's, and the operand carries u = s A x after x.
// Cross-wave partial sums meet in LDS; the epilogue runs on the reduced tile.
// ---------------------------------------------------------------------------
template <typename T, int EPI, int MG, bool SPLIT>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
    constexpr int FK = Elt<T>::FK;
    constexpr int EPL = Elt<T>::EPL;
    // fragments in flight per wave (register budget: W, X and X residual)
    constexpr int UNR = SPLIT ? ((MG >= 8) ? 1 : (MG >= 4 ? 2 : 4)) : ((MG >= 8) ? 2 : (MG >= 4 ? 4 : 8));
    __shared__ f32x4 s_red[4][MG][WAVE];
    __shared__ float s_tile[MG][16][17];

    const int lane = threadIdx.x % WAVE;
    const int wid = threadIdx.x / WAVE;
    const int tile = blockIdx.x / a.ks;
    const int split = blockIdx.x % a.ks;
    const int fps = a.kb / a.ks;
    const int f_begin = split * fps;
    const int n_tail = (split == a.ks - 1) ? a.tail_frags : 0;
    const int nf = fps + n_tail;
    const int lrow = lane % 16, lgrp = lane / 16;

    // Operand sources of the LoRA tail.
    const uint4* xt0 = a.xt[0];
    const uint4* xt1 = a.xt[1];
    if (a.tail_mode == TAIL_BY_TILE) {
        xt0 = tile < a.tile_split0 ? a.xt[0] : (tile < a.tile_split1 ? a.xt[1] : a.xt[2]);
    }
    const uint4* wt = a.w + (size_t)tile * a.ft * WAVE;

    for (int mg0 = 0; mg0 < a.MT; mg0 += MG) {
        const int mgn = min(MG, a.MT - mg0);
        f32x4 acc[MG];
#pragma unroll
        for (int i = 0; i < MG; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

        for (int base = wid; base < nf; base += 4 * UNR) {
            uint4 wv[UNR];
            uint4 xv[UNR][MG];
            uint4 xv2[UNR][MG];     // tail: second source; base: operand residual (SPLIT)
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int i = base + 4 * u;
                wv[u] = uint4{0, 0, 0, 0};
#pragma unroll
                for (int mt = 0; mt < MG; ++mt) { xv[u][mt] = uint4{0, 0, 0, 0}; xv2[u][mt] = uint4{0, 0, 0, 0}; }
                if (i < nf) {
                    const bool is_tail = i >= fps;
                    const int f = is_tail ? (a.kb + i - fps) : (f_begin + i);
                    const int tf = i - fps;
                    const bool lane_live = !is_tail || (tf * FK + lgrp * EPL < a.r);
                    if (lane_live) wv[u] = wt[(size_t)f * WAVE + lane];
#pragma unroll
                    for (int mt = 0; mt < MG; ++mt) {
                        const int m = (mg0 + mt) * 16 + lrow;
                        if (mt < mgn && m < a.M) {
                            if (!is_tail) {
                                xv[u][mt] = a.x[((size_t)f * a.MT + mg0 + mt) * WAVE + lane];
                                if (SPLIT) xv2[u][mt] = a.xlo[((size_t)f * a.MT + mg0 + mt) * WAVE + lane];
                            } else {
                                xv[u][mt] = xt0[((size_t)tf * a.MT + mg0 + mt) * WAVE + lane];
                                if (a.tail_mode == TAIL_BY_ROW_HALF)
                                    xv2[u][mt] = xt1[((size_t)tf * a.MT + mg0 + mt) * WAVE + lane];
                            }
                        }
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int i = base + 4 * u;
                if (i < nf) {
                    if (a.tail_mode == TAIL_BY_ROW_HALF && i >= fps) {
                        // rows 0-7 of the tile use source 0, rows 8-15 source 1
                        const uint4 zero = uint4{0, 0, 0, 0};
                        const uint4 w_lo = lrow < 8 ? wv[u] : zero;
                        const uint4 w_hi = lrow < 8 ? zero : wv[u];
#pragma unroll
                        for (int mt = 0; mt < MG; ++mt) {
                            mma_frag<T>(acc[mt], w_lo, xv[u][mt]);
                            mma_frag<T>(acc[mt], w_hi, xv2[u][mt]);
                        }
                    } else {
#pragma unroll
                        for (int mt = 0; mt < MG; ++mt) {
                            mma_frag<T>(acc[mt], wv[u], xv[u][mt]);
                            if (SPLIT && i < fps) mma_frag<T>(acc[mt], wv[u], xv2[u][mt]);
                        }
                    }
                }
            }
        }

        // Reduce the four waves' partial tiles (fixed order).
#pragma unroll
        for (int mt = 0; mt < MG; ++mt) s_red[wid][mt][lane] = acc[mt];
        __syncthreads();
        for (int idx = threadIdx.x; idx < MG * WAVE * 4; idx += blockDim.x) {
            const int mt = idx / (WAVE * 4);
            const int ln = (idx / 4) % WAVE;
            const int e = idx % 4;
            float v = s_red[0][mt][ln][e] + s_red[1][mt][ln][e] + s_red[2][mt][ln][e] + s_red[3][mt][ln][e];
            s_tile[mt][(ln / 16) * 4 + e][ln % 16] = v;    // [n in tile][m in tile]
        }
        __syncthreads();

        // Epilogues.
        if (EPI == EPI_STORE) {
            // out[m][n0 + n] (fp32, row stride ldo), for the QKV projection
            for (int idx = threadIdx.x; idx < mgn * 256; idx += blockDim.x) {
                const int mt = idx / 256, n = idx % 16, ml = (idx / 16) % 16;
                const int m = (mg0 + mt) * 16 + ml;
                if (m < a.M) a.out[(size_t)m * a.ldo + tile * 16 + n] = s_tile[mt][n][ml];
            }
        } else if (EPI == EPI_PARTIAL) {
            // split-K partial sums, folded in order by the next k_norm
            float* o = a.out + (size_t)split * a.partial_stride;
            for (int idx = threadIdx.x; idx < mgn * 256; idx += blockDim.x) {
                const int mt = idx / 256, n = idx % 16, ml = (idx / 16) % 16;
                const int m = (mg0 + mt) * 16 + ml;
                if (m < a.M) o[(size_t)m * a.ldo + tile * 16 + n] = s_tile[mt][n][ml];
            }
        } else if (EPI == EPI_SWIGLU) {
            // tile rows 0-7: gate rows 8*tile..; rows 8-15: the matching up rows.
            T* h = (T*)a.out_frag;
            for (int idx = threadIdx.x; idx < mgn * 128; idx += blockDim.x) {
                const int mt = idx / 128, c = idx % 8, ml = (idx / 8) % 16;
                const int m = (mg0 + mt) * 16 + ml;
                if (m < a.M) {
                    const float gt = s_tile[mt][c][ml];
                    const float up = s_tile[mt][c + 8][ml];
                    const float hv = gt / (1.f + __expf(-gt)) * up;
                    const T hq = from_f32<T>(hv);
                    const size_t e = xfrag_elem<T>(m, tile * 8 + c, a.out_MT);
                    h[e] = hq;
                    if (SPLIT) ((T*)a.out_frag_lo)[e] = from_f32<T>(hv - to_f32(hq));
                }
            }
        } else {  // EPI_ARGMAX: tied LM head, per-tile (max, argmax) per row
            for (int idx = threadIdx.x; idx < mgn * 16; idx += blockDim.x) {
                const int mt = idx / 16, ml = idx % 16;
                const int m = (mg0 + mt) * 16 + ml;
                if (m >= a.M) continue;
                float best = -INFINITY;
                int bi = 0x7fffffff;
                for (int n = 0; n < 16; ++n) {
                    const int v = tile * 16 + n;
                    const float val = s_tile[mt][n][ml];
                    if (a.logits) a.logits[(size_t)m * a.ldo + v] = val;
                    if (v == a.exclude) continue;
                    if (val > best) { best = val; bi = v; }   // ascending v: first max wins ties
                }
                a.arg_val[(size_t)tile * a.M + m] = best;
                a.arg_idx[(size_t)tile * a.M + m] = bi;
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Split-KV attention on MFMA
//
// Work item (split s, KV head g, sequence b): the G = h_q / h_kv query heads of
// g over the W block rows (QR = G*W query rows, QT tiles of 16) against prefix
// keys [k_lo, k_hi) and, in the last split, the W block keys.  S^T = K Q^T is
// computed per 16-key block (A = K fragment from the cache, B = Q^T kept in
// registers), softmax runs online per query column in the exp2 domain, and
// O^T += V^T P^T takes P^T directly from the score accumulators.
// ---------------------------------------------------------------------------
template <typename T, int HD, int QT>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
    constexpr int FK = Elt<T>::FK;
    constexpr int EPL = Elt<T>::EPL;
    constexpr int NDS = HD / FK;          // fragments per key row
    constexpr int NDT = HD / 16;          // V^T tiles
    constexpr int QROWS = QT * 16;
    constexpr int LDQ = HD + 16 / (int)sizeof(T);   // padded LDS row (bank spread)
    constexpr int KBMAX = 48;                       // block keys: W <= 33 -> 3 blocks
    typedef typename K4<T>::raw vraw;

    const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int t = a.pos0[b];
    const int nrows = a.nrows[b];
    int s_eff, chunk;
    attn_splits(t, a.kps, a.s_launch, s_eff, chunk);
    if (s >= s_eff) return;
    const int k_lo = min(s * chunk, t);
    const int k_hi = min(t, k_lo + chunk);
    const bool last = (s == s_eff - 1);
    const int W = a.W, G = a.G;
    const int QR = G * W;

    extern __shared__ __align__(16) unsigned char smem[];
    T* q_l = (T*)smem;                                   // [QROWS][LDQ]
    T* kb_l = q_l + QROWS * LDQ;                         // [KBMAX][LDQ]
    T* vb_l = kb_l + KBMAX * LDQ;                        // [KBMAX][HD]
    float* obuf = (float*)smem;                          // [QROWS][HD] (aliases after the loop)
    float* ml_l = (float*)(smem + a.smem_main);          // [4][QROWS][2]

    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    const int lrow = lane % 16, lgrp = lane / 16;
    const size_t row_stride = (size_t)a.nqkv;
    const float* qkv_b = a.qkv + (size_t)b * W * row_stride;

    // -- Q: per-head RMSNorm, RoPE at position t + j, rounded to T (one wave per row)
    const T* gq = (const T*)a.q_norm;
    const T* gk = (const T*)a.k_norm;
    const float2* rope = a.rope;
    for (int q = wid; q < QROWS; q += 4) {
        T* dst = q_l + q * LDQ;
        if (q >= QR) {
            for (int i = lane; i < HD; i += WAVE) dst[i] = from_f32<T>(0.f);
            continue;
        }
        const int gi = q / W, j = q % W;
        const float* src = qkv_b + (size_t)j * row_stride + (size_t)(g * G + gi) * HD;
        const int half = HD / 2;
        float x0 = lane < half ? src[lane] : 0.f;
        float x1 = lane < half ? src[lane + half] : 0.f;
        float inv = 1.f;
        if (a.qk_norm) {
            float ss = wave_sum(x0 * x0 + x1 * x1);
            inv = rsqrtf(ss / (float)HD + a.eps);
        }
        if (lane < half) {
            float y0 = x0 * inv, y1 = x1 * inv;
            if (a.qk_norm) { y0 *= to_f32(gq[lane]); y1 *= to_f32(gq[lane + half]); }
            const float2 cs = rope[(size_t)(t + j) * half + lane];
            dst[lane] = from_f32<T>(y0 * cs.x - y1 * cs.y);
            dst[lane + half] = from_f32<T>(y1 * cs.x + y0 * cs.y);
        }
    }
    // -- block keys and values (last split only); the verify appends them to the cache
    const int nkb_blk = last ? ceil_div(W, 16) : 0;
    T* kc = (T*)a.kcache + (((size_t)a.layer * a.max_batch + b) * a.n_kv + g) * a.nblk * 16 * HD;
    T* vc = (T*)a.vcache + (((size_t)a.layer * a.max_batch + b) * a.n_kv + g) * a.nblk * 16 * HD;
    if (last) {
        for (int j = wid; j < nkb_blk * 16; j += 4) {
            T* kd = kb_l + j * LDQ;
            T* vd = vb_l + j * HD;
            if (j >= W || j >= nrows) {
                for (int i = lane; i < HD; i += WAVE) { kd[i] = from_f32<T>(0.f); vd[i] = from_f32<T>(0.f); }
                continue;
            }
            const float* ks = qkv_b + (size_t)j * row_stride + (size_t)a.n_q * HD + (size_t)g * HD;
            const float* vs = ks + (size_t)a.n_kv * HD;
            const int half = HD / 2;
            float x0 = lane < half ? ks[lane] : 0.f;
            float x1 = lane < half ? ks[lane + half] : 0.f;
            float inv = 1.f;
            if (a.qk_norm) {
                float ss = wave_sum(x0 * x0 + x1 * x1);
                inv = rsqrtf(ss / (float)HD + a.eps);
            }
            const int pos = t + j;
            if (lane < half) {
                float y0 = x0 * inv, y1 = x1 * inv;
                if (a.qk_norm) { y0 *= to_f32(gk[lane]); y1 *= to_f32(gk[lane + half]); }
                const float2 cs = rope[(size_t)pos * half + lane];
                const T k0 = from_f32<T>(y0 * cs.x - y1 * cs.y);
                const T k1 = from_f32<T>(y1 * cs.x + y0 * cs.y);
                kd[lane] = k0;
                kd[lane + half] = k1;
                if (a.write_kv) {
                    T* blk = kc + (size_t)(pos / 16) * 16 * HD;
                    blk[kblock_elem<T>(pos % 16, lane)] = k0;
                    blk[kblock_elem<T>(pos % 16, lane + half)] = k1;
                }
            }
            for (int i = lane; i < HD; i += WAVE) {
                const T v = from_f32<T>(vs[i]);
                vd[i] = v;
                if (a.write_kv) vc[(size_t)(pos / 16) * 16 * HD + vblock_elem(pos % 16, i)] = v;
            }
        }
    }
    __syncthreads();

    // -- Q^T fragments in registers
    uint4 qf[QT][NDS];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds)
            qf[qt][ds] = *(const uint4*)(q_l + (qt * 16 + lrow) * LDQ + ds * FK + lgrp * EPL);

    // block row of each of this lane's query columns (for the causal mask)
    int jq[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) jq[qt] = (qt * 16 + lrow) % W;

    f32x4 o_acc[NDT][QT];
    float m_run[QT], l_run[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m_run[qt] = -1e30f;
        l_run[qt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o_acc[dt][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    const int kb_first = k_lo / 16;
    const int n_pref = (k_hi > k_lo) ? ceil_div(k_hi, 16) - kb_first : 0;
    const int n_items = n_pref + nkb_blk;
    const float sl2 = a.scale_log2;

    for (int it = wid; it < n_items; it += 4) {
        const bool pref = it < n_pref;
        uint4 kf[NDS];
        vraw vf[NDT];
        int key0;
        if (pref) {
            const int kb = kb_first + it;
            key0 = kb * 16;
            const T* kblk = kc + (size_t)kb * 16 * HD;
            const T* vblk = vc + (size_t)kb * 16 * HD;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) kf[ds] = *(const uint4*)(kblk + (size_t)(ds * WAVE + lane) * EPL);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) vf[dt] = *(const vraw*)(vblk + (size_t)(dt * WAVE + lane) * 4);
        } else {
            const int bb = it - n_pref;
            key0 = bb * 16;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                kf[ds] = *(const uint4*)(kb_l + (bb * 16 + lrow) * LDQ + ds * FK + lgrp * EPL);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                T tmp[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) tmp[e] = vb_l[(bb * 16 + lgrp * 4 + e) * HD + dt * 16 + lrow];
                __builtin_memcpy(&vf[dt], tmp, sizeof(vraw));
            }
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) mma_frag<T>(sc, kf[ds], qf[qt][ds]);
            // lane holds keys key0 + 4*lgrp + e for query column qt*16 + lrow
            float sv[4];
            bool valid[4];
            float mloc = -1e30f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int kk = key0 + lgrp * 4 + e;
                bool ok;
                if (pref) ok = kk < k_hi;
                else ok = kk < nrows && (!a.causal || kk <= jq[qt]);
                valid[e] = ok;
                sv[e] = sc[e] * sl2;
                if (ok) mloc = fmaxf(mloc, sv[e]);
            }
            mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
            mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
            const float m_new = fmaxf(m_run[qt], mloc);
            const float corr = exp2f(m_run[qt] - m_new);
            f32x4 p;
            float psum = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                p[e] = valid[e] ? exp2f(sv[e] - m_new) : 0.f;
                psum += p[e];
            }
            psum += __shfl_xor(psum, 16, 64);
            psum += __shfl_xor(psum, 32, 64);
            l_run[qt] = l_run[qt] * corr + psum;
            m_run[qt] = m_new;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                o_acc[dt][qt] *= corr;
                mma_k4(o_acc[dt][qt], vf[dt], p);
            }
        }
    }

    // -- merge the four waves (fixed order) and write this split's partial
    __syncthreads();                                     // LDS operands dead: obuf may alias
    if (lgrp == 0) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            ml_l[(wid * QROWS + qt * 16 + lrow) * 2 + 0] = m_run[qt];
            ml_l[(wid * QROWS + qt * 16 + lrow) * 2 + 1] = l_run[qt];
        }
    }
    __syncthreads();
    float fct[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int q = qt * 16 + lrow;
        float mx = -1e30f;
        for (int w = 0; w < 4; ++w) mx = fmaxf(mx, ml_l[(w * QROWS + q) * 2]);
        fct[qt] = exp2f(m_run[qt] - mx);
    }
    for (int w = 0; w < 4; ++w) {
        if (wid == w) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt)
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int d = dt * 16 + lgrp * 4 + e;
                        const int q = qt * 16 + lrow;
                        const float v = o_acc[dt][qt][e] * fct[qt];
                        if (w == 0) obuf[q * HD + d] = v;
                        else obuf[q * HD + d] += v;
                    }
        }
        __syncthreads();
    }
    // partial (max in log2 domain, sum, unnormalised output) per query row
    const int S = a.s_launch;
    for (int idx = threadIdx.x; idx < QR * HD; idx += blockDim.x) {
        const int q = idx / HD, d = idx % HD;
        const int gi = q / W, j = q % W;
        const size_t pr = (((size_t)b * a.n_q + g * G + gi) * W + j) * S + s;
        a.part_o[pr * HD + d] = obuf[q * HD + d];
    }
    for (int q = threadIdx.x; q < QR; q += blockDim.x) {
        float mx = -1e30f;
        for (int w = 0; w < 4; ++w) mx = fmaxf(mx, ml_l[(w * QROWS + q) * 2]);
        float L = 0.f;
        for (int w = 0; w < 4; ++w) L += ml_l[(w * QROWS + q) * 2 + 1] * exp2f(ml_l[(w * QROWS + q) * 2] - mx);
        const int gi = q / W, j = q % W;
        const size_t pr = (((size_t)b * a.n_q + g * G + gi) * W + j) * S + s;
        a.part_ml[pr * 2 + 0] = mx;
        a.part_ml[pr * 2 + 1] = L;
    }
}

// Merge the split-KV partials of one block row for every query head, write the
// O-projection operand, and (draft) its LoRA shrink.
template <typename T>
__global__ __launch_bounds__(256) void k_combine(CombineArgs a) {
    const int m = blockIdx.x;
    const int b = m / a.W, j = m % a.W;
    const int HD = a.head_dim, NQ = a.n_q;
    const int K = NQ * HD;
    __shared__ float s_o[MAX_SHRINK_DIM];
    int s_eff, chunk;
    attn_splits(a.pos0[b], a.kps, a.s_launch, s_eff, chunk);
    const int S = a.s_launch;
    T* xf = (T*)a.xfrag;
    for (int idx = threadIdx.x; idx < K; idx += blockDim.x) {
        const int h = idx / HD, d = idx % HD;
        const size_t pr0 = (((size_t)b * NQ + h) * a.W + j) * S;
        float mx = -1e30f;
        for (int s = 0; s < s_eff; ++s) mx = fmaxf(mx, a.part_ml[(pr0 + s) * 2]);
        float L = 0.f, o = 0.f;
        for (int s = 0; s < s_eff; ++s) {
            const float wgt = exp2f(a.part_ml[(pr0 + s) * 2] - mx);
            L += wgt * a.part_ml[(pr0 + s) * 2 + 1];
            o += wgt * a.part_o[(pr0 + s) * HD + d];
        }
        const float val = (L > 0.f) ? o / L : 0.f;
        const T q = from_f32<T>(val);
        const size_t e = xfrag_elem<T>(m, idx, a.MT);
        xf[e] = q;
        if (a.xfrag_lo) ((T*)a.xfrag_lo)[e] = from_f32<T>(val - to_f32(q));
        s_o[idx] = a.xfrag_lo ? val : to_f32(q);
    }
    if (a.r == 0 || a.lora_a == nullptr) return;
    __syncthreads();
    const int wid = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
    for (int jj = wid; jj < a.r; jj += blockDim.x / WAVE) {
        const T* A = (const T*)a.lora_a + (size_t)jj * K;
        float acc = 0.f;
        for (int k = lane; k < K; k += WAVE) acc += to_f32(A[k]) * s_o[k];
        acc = wave_sum(acc);
        if (lane == 0) ((T*)a.tail)[xfrag_elem<T>(m, jj, a.MT)] = from_f32<T>(acc * a.scale);
    }
}

// ---------------------------------------------------------------------------
// Final argmax over the LM-head tile partials (ties: lowest id) and routing of
// the result: draft tokens (rows 1..D), verify tokens (rows 0..D), or the
// prefill's first generated token.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_argmax(ArgmaxArgs a) {
    const int m = blockIdx.x;
    const int b = m / a.W, j = m % a.W;
    float best = -INFINITY;
    int bi = 0x7fffffff;
    for (int tI = threadIdx.x; tI < a.n_tiles; tI += blockDim.x) {
        const float v = a.arg_val[(size_t)tI * a.M + m];
        const int i = a.arg_idx[(size_t)tI * a.M + m];
        if (v > best || (v == best && i < bi)) { best = v; bi = i; }
    }
    __shared__ float s_v[256];
    __shared__ int s_i[256];
    s_v[threadIdx.x] = best;
    s_i[threadIdx.x] = bi;
    __syncthreads();
    for (int st = blockDim.x / 2; st > 0; st >>= 1) {
        if ((int)threadIdx.x < st) {
            const float v2 = s_v[threadIdx.x + st];
            const int i2 = s_i[threadIdx.x + st];
            if (v2 > s_v[threadIdx.x] || (v2 == s_v[threadIdx.x] && i2 < s_i[threadIdx.x])) {
                s_v[threadIdx.x] = v2;
                s_i[threadIdx.x] = i2;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    const int tok = s_i[0];
    if (a.mode == PASS_DRAFT) {
        if (j >= 1) a.out[b * (a.W - 1) + j - 1] = tok;
    } else if (a.mode == PASS_VERIFY) {
        a.out[b * a.W + j] = tok;
    } else {
        if (a.chunk_pos + j == a.lengths[b] - 1 && j < a.nrows[b]) {
            a.out[b] = tok;                     // anchor
            a.seq_len_out[b] = a.lengths[b];
        }
    }
}

// Longest-prefix acceptance and commit (Sec. 3 steps 4-5, App. A.1).
__global__ void k_accept(AcceptArgs a) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= a.B) return;
    const int D = a.D, W = D + 1;
    const int t = a.seq_len[b];
    int n = 0;
    if (a.forced) {
        n = a.forced[b];
        if (n < 0 || n > D) { atomicOr(a.status, PBD_STATUS_FORCED_N); return; }
    } else {
        while (n < D && a.draft[b * D + n] == a.verify[b * W + n]) ++n;
    }
    if (t < 0 || t + n + 1 > a.max_seq) { atomicOr(a.status, PBD_STATUS_CAPACITY); return; }
    for (int i = 0; i < W; ++i)
        a.out[b * W + i] = i < n ? a.draft[b * D + i] : (i == n ? a.verify[b * W + n] : -1);
    a.n_acc[b] = n;
    a.seq_len[b] = t + n + 1;
    a.anchor[b] = a.verify[b * W + n];
}

// ---------------------------------------------------------------------------
// Initialisation helpers
// ---------------------------------------------------------------------------
// Repack [rows][K] weights (+ LoRA B [rows][r]) into 16-row fragment tiles.
template <typename T>
__global__ void k_pack(PackArgs a) {
    constexpr int EPL = Elt<T>::EPL;
    constexpr int FK = Elt<T>::FK;
    const size_t total = (size_t)a.n_tiles * a.ft * WAVE;
    for (size_t id = blockIdx.x * (size_t)blockDim.x + threadIdx.x; id < total; id += (size_t)gridDim.x * blockDim.x) {
        const int lane = id % WAVE;
        const int f = (id / WAVE) % a.ft;
        const int tile = id / ((size_t)WAVE * a.ft);
        const int row = lane % 16, grp = lane / 16;
        int src, srow;
        if (a.row_map == MAP_INTERLEAVE2) {
            src = row < 8 ? 0 : 1;
            srow = tile * 8 + (row % 8);
        } else {
            const int r = tile * 16 + row;
            src = 0;
            srow = r;
            if (a.n_src > 1 && r >= a.src_rows[0]) { src = 1; srow = r - a.src_rows[0]; }
            if (a.n_src > 2 && r >= a.src_rows[0] + a.src_rows[1]) { src = 2; srow = r - a.src_rows[0] - a.src_rows[1]; }
        }
        T vals[EPL];
        if (f < a.kb) {
            const T* Wsrc = (const T*)a.w[src] + (size_t)srow * a.K + f * FK + grp * EPL;
#pragma unroll
            for (int e = 0; e < EPL; ++e) vals[e] = Wsrc[e];
        } else {
            const int kt = (f - a.kb) * FK + grp * EPL;
#pragma unroll
            for (int e = 0; e < EPL; ++e)
                vals[e] = (a.b[src] && kt + e < a.r) ? ((const T*)a.b[src])[(size_t)srow * a.r + kt + e] : from_f32<T>(0.f);
        }
        T* dst = (T*)a.dst + id * EPL;
#pragma unroll
        for (int e = 0; e < EPL; ++e) dst[e] = vals[e];
    }
}

__global__ void k_fill_u32(uint32_t* p, size_t n, uint32_t v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------
template <typename T, bool SPLIT>
static hipError_t launch_gemm_t(const GemmArgs& a, int epi, hipStream_t st) {
    const int mg = a.MT <= 1 ? 1 : (a.MT <= 2 ? 2 : (a.MT <= 4 ? 4 : 8));
    dim3 grid(a.n_tiles * a.ks), block(256);
#define PBD_GEMM_CASE(E, G)                                                     \
    if (epi == E && mg == G) { hipLaunchKernelGGL((k_gemm<T, E, G, SPLIT>), grid, block, 0, st, a); return hipGetLastError(); }
#define PBD_GEMM_EPI(E) PBD_GEMM_CASE(E, 1) PBD_GEMM_CASE(E, 2) PBD_GEMM_CASE(E, 4) PBD_GEMM_CASE(E, 8)
    PBD_GEMM_EPI(EPI_STORE)
    PBD_GEMM_EPI(EPI_PARTIAL)
    PBD_GEMM_EPI(EPI_SWIGLU)
    PBD_GEMM_EPI(EPI_ARGMAX)
#undef PBD_GEMM_EPI
#undef PBD_GEMM_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_gemm(int dtype, const GemmArgs& a, int epi, hipStream_t st) {
    if (dtype == PBD_DTYPE_BF16)
        return a.xlo ? launch_gemm_t<bf16, true>(a, epi, st) : launch_gemm_t<bf16, false>(a, epi, st);
    return launch_gemm_t<float, false>(a, epi, st);
}

size_t attn_smem_main(int dtype, int head_dim, int qt) {
    const size_t es = dtype == PBD_DTYPE_BF16 ? 2 : 4;
    const size_t ldq = head_dim + 16 / es;
    const size_t ops = (qt * 16 * ldq + 48 * ldq + 48 * (size_t)head_dim) * es;
    const size_t ob = (size_t)qt * 16 * head_dim * 4;
    size_t m = ops > ob ? ops : ob;
    return (m + 15) / 16 * 16;
}

size_t attn_smem_bytes(int dtype, int head_dim, int qt) {
    return attn_smem_main(dtype, head_dim, qt) + (size_t)4 * qt * 16 * 2 * 4;
}

template <typename T, int HD>
static hipError_t launch_attn_hd(const AttnArgs& a, int qt, dim3 grid, size_t smem, hipStream_t st) {
    switch (qt) {
        case 1: hipLaunchKernelGGL((k_attn<T, HD, 1>), grid, dim3(256), smem, st, a); break;
        case 2: hipLaunchKernelGGL((k_attn<T, HD, 2>), grid, dim3(256), smem, st, a); break;
        case 3: hipLaunchKernelGGL((k_attn<T, HD, 3>), grid, dim3(256), smem, st, a); break;
        case 4: hipLaunchKernelGGL((k_attn<T, HD, 4>), grid, dim3(256), smem, st, a); break;
        case 5: hipLaunchKernelGGL((k_attn<T, HD, 5>), grid, dim3(256), smem, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attn(int dtype, int head_dim, int qt, const AttnArgs& a, int batch, hipStream_t st) {
    dim3 grid(a.s_launch, a.n_kv, batch);
    const size_t smem = attn_smem_bytes(dtype, head_dim, qt);
    if (dtype == PBD_DTYPE_BF16) {
        if (head_dim == 128) return launch_attn_hd<bf16, 128>(a, qt, grid, smem, st);
        if (head_dim == 64) return launch_attn_hd<bf16, 64>(a, qt, grid, smem, st);
    } else {
        if (head_dim == 128) return launch_attn_hd<float, 128>(a, qt, grid, smem, st);
        if (head_dim == 64) return launch_attn_hd<float, 64>(a, qt, grid, smem, st);
    }
    return hipErrorInvalidValue;
}

#define PBD_DISPATCH(dtype, KERNEL, grid, block, st, args)                                   \
    do {                                                                                     \
        if ((dtype) == PBD_DTYPE_BF16) hipLaunchKernelGGL(KERNEL<bf16>, grid, block, 0, st, args); \
        else hipLaunchKernelGGL(KERNEL<float>, grid, block, 0, st, args);                    \
        return hipGetLastError();                                                            \
    } while (0)

hipError_t launch_assemble(int dtype, const AssembleArgs& a, int batch, hipStream_t st) {
    PBD_DISPATCH(dtype, k_assemble, dim3(batch), dim3(256), st, a);
}
hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st) {
    PBD_DISPATCH(dtype, k_norm, dim3(a.M), dim3(256), st, a);
}
hipError_t launch_shrink(int dtype, const ShrinkArgs& a, hipStream_t st) {
    PBD_DISPATCH(dtype, k_shrink, dim3(a.M), dim3(256), st, a);
}
hipError_t launch_combine(int dtype, const CombineArgs& a, hipStream_t st) {
    PBD_DISPATCH(dtype, k_combine, dim3(a.M), dim3(256), st, a);
}
hipError_t launch_pack(int dtype, const PackArgs& a, hipStream_t st) {
    PBD_DISPATCH(dtype, k_pack, dim3(1024), dim3(256), st, a);
}
hipError_t launch_argmax(const ArgmaxArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(k_argmax, dim3(a.M), dim3(256), 0, st, a);
    return hipGetLastError();
}
hipError_t launch_accept(const AcceptArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(k_accept, dim3((a.B + 63) / 64), dim3(64), 0, st, a);
    return hipGetLastError();
}
hipError_t launch_fill_u32(void* p, size_t n_words, uint32_t v, hipStream_t st) {
    if (n_words == 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_u32, dim3(1024), dim3(256), 0, st, (uint32_t*)p, n_words, v);
    return hipGetLastError();
}

}  // namespace pbd
