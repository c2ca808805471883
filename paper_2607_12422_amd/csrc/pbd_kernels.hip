// HIP kernels of the PEFT-BD speculative step for gfx950.
//
// One pass (draft or verify, Sec. 3 steps 1-3) runs six kernels per layer:
//   k_fgemm<STORE>   q/k/v projection; RMSNorm folded in as a per-row scale of the
//                    accumulator; LoRA shrink A x and expand B u inside the tile
//                    (App. A.2) when the adapter is on
//   k_attn           split-KV attention partials on MFMA over the committed prefix
//                    and the block (bidirectional or causal block mask); QK-norm and
//                    RoPE of the block rows; the verify appends the block K/V
//   k_combine        merge the split partials into the O-projection operand
//   k_fgemm<RESID>   O projection + LoRA + residual add; writes the next RMSNorm's
//                    operand and per-row sums of squares
//   k_fgemm<SWIGLU>  gate/up projection + LoRA, SwiGLU epilogue
//   k_fgemm<RESID>   down projection + LoRA + residual add
// then the tied LM head with a fused argmax, and the longest-prefix acceptance
// (Sec. 3 step 4, App. A.1).
//
// RMSNorm by linearity: W (x / rms(x) * g) = r_m * W (x * g) with r_m = 1 / rms
// of row m, so producers write x * g and sum(x^2) partials, and consumers scale
// their accumulators by r_m; no standalone normalisation kernel runs.
#include "pbd_device.h"
#include <hip/hip_ext.h>

#include "pbd_kernels.h"

#include <algorithm>

namespace pbd {

// Optional timing events attached to the next launch (profiling aid): with
// events set, kernels are launched with hipExtLaunchKernel, whose events carry
// the dispatch's own start and end times.
static thread_local hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;
void set_launch_events(hipEvent_t start, hipEvent_t stop) {
    g_ev_start = start;
    g_ev_stop = stop;
}
void get_launch_events(hipEvent_t* start, hipEvent_t* stop) {
    *start = g_ev_start;
    *stop = g_ev_stop;
}
#define PBD_LAUNCH(KERNEL, GRID, BLOCK, SHMEM, ST, ...)                                              \
    do {                                                                                            \
        if (g_ev_start)                                                                             \
            hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, ST, g_ev_start, g_ev_stop, 0, __VA_ARGS__); \
        else                                                                                        \
            hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, ST, __VA_ARGS__);                        \
    } while (0)

static __device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Split-KV schedule shared by k_attn and k_combine: prefix splits s < s_pre
// cover keys [0, t) in chunks of `chunk` keys (a multiple of 16); split s_pre
// holds the W block keys.  s_launch >= 2.
static __device__ __forceinline__ void attn_splits(int t, int kps, int s_launch, int& s_pre, int& chunk) {
    s_pre = t > 0 ? min(ceil_div(t, kps), s_launch - 1) : 0;
    chunk = s_pre > 0 ? ceil_div(ceil_div(t, s_pre), 16) * 16 : 16;
}

// Write EPL consecutive k values of one operand row (16-byte aligned run of
// one lane's fragment slot) as value and residual, or plain T when lo is null;
// with h16 (bf16 models only) as fp16 values into hi.
template <typename T>
static __device__ __forceinline__ void put_operand_run(T* hi, T* lo, size_t e, const float* v, bool h16 = false) {
    constexpr int EPL = Elt<T>::EPL;
    if constexpr (EPL == 8) {
        if (h16) {
            _Float16 hh[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) hh[i] = (_Float16)v[i];
            uint4 hv;
            __builtin_memcpy(&hv, hh, 16);
            *(uint4*)(hi + e) = hv;
            return;
        }
    }
    T h[EPL], l[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        h[i] = from_f32<T>(v[i]);
        l[i] = from_f32<T>(v[i] - to_f32(h[i]));
    }
    uint4 hv, lv;
    __builtin_memcpy(&hv, h, 16);
    __builtin_memcpy(&lv, l, 16);
    *(uint4*)(hi + e) = hv;
    if (lo) *(uint4*)(lo + e) = lv;
}

// Write v into an operand as bf16 value (hi) plus bf16 residual (lo), or as
// plain T when lo is null.
template <typename T>
static __device__ __forceinline__ void put_operand(T* hi, T* lo, size_t e, float v) {
    const T h = from_f32<T>(v);
    hi[e] = h;
    if (lo) lo[e] = from_f32<T>(v - to_f32(h));
}

// ---------------------------------------------------------------------------
// Block assembly and embedding gather (Sec. 3 steps 1 and 3); writes the
// residual x, the first q/k/v operand x * g and per-row sums of squares.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_assemble(AssembleArgs a) {
    const int j = blockIdx.x, b = blockIdx.y;
    const int W = a.W;
    // sequence state: every row's work-group derives the same values
    int pos0, nrows;
    bool ok = true;
    if (a.mode == PASS_PREFILL) {
        const int len = a.lengths[b];
        if (len < 1 || len > a.max_len || len + a.room > a.max_seq) ok = false;
        pos0 = a.chunk_pos;
        nrows = ok ? min(max(len - a.chunk_pos, 0), W) : 0;
    } else {
        pos0 = a.seq_len[b] + a.pos_add;
        if (pos0 < 0 || pos0 + W > a.max_seq) ok = false;
        nrows = ok ? W : 0;
    }
    if (!ok) pos0 = 0;
    int tok;
    const int nd = W - a.lead;
    if (a.mode == PASS_PREFILL) tok = (j < nrows) ? a.prompt[(size_t)b * a.max_len + a.chunk_pos + j] : 0;
    else if (j < a.lead) tok = a.anchor[b];
    else if (a.mode == PASS_DRAFT) tok = a.drafts ? a.drafts[b * nd + j - a.lead] : a.mask_id;
    else tok = a.drafts[b * nd + j - a.lead];
    const bool bad_tok = tok < 0 || tok >= a.vocab;
    if (bad_tok) tok = 0;
    if (threadIdx.x == 0 && a.fused_ctl && j == 0 && b == 0) {
        // the persistent pass that follows reads these when it starts
        for (int i = 0; i < 8; ++i) a.fused_ctl[i] = 0u;
        a.fused_ctl[8] += 1u;
        a.fused_ctl[9] = 0u;
        // writes so far into each layer-parity half of its partial buffers:
        // the pass reads the counts before it and (unless the sequence is
        // skipped, when it writes nothing) they advance by its layers of each parity
        if (nrows > 0) {
            a.fused_ctl[14] = a.fused_ctl[12];
            a.fused_ctl[15] = a.fused_ctl[13];
            a.fused_ctl[12] += (unsigned)((a.fused_layers + 1) / 2);
            a.fused_ctl[13] += (unsigned)(a.fused_layers / 2);
        }
    }
    if (threadIdx.x == 0) {
        if (j == 0) {
            a.pos0[b] = pos0;
            a.nrows[b] = nrows;
            if (!ok) atomicOr(a.status, PBD_STATUS_CAPACITY);
        }
        if (bad_tok && j < nrows) atomicOr(a.status, PBD_STATUS_TOKEN);
        a.tokens[b * W + j] = tok;
    }
    // gather the embedding row from the fragment-packed table: one 16-byte
    // chunk of EPL consecutive features per thread and step
    constexpr int EPL = Elt<T>::EPL;
    constexpr int FK = Elt<T>::FK;
    const T* E = (const T*)a.embed;
    const T* g = (const T*)a.gain;
    const int m = b * W + j;
    const int ft = a.H / FK;
    const int nchunk = a.H / EPL;
    float ss = 0.f;
    for (int c = threadIdx.x; c < nchunk; c += blockDim.x) {
        const int k0 = c * EPL;
        const uint4 raw = *(const uint4*)(E + frag_elem<T>((size_t)(tok / 16) * ft + k0 / FK, tok % 16, k0 % FK));
        const T* v = (const T*)&raw;
        float xv[EPL];
#pragma unroll
        for (int e = 0; e < EPL; ++e) xv[e] = to_f32(v[e]);
        *(float4*)(a.x + (size_t)m * a.H + k0) = float4{xv[0], xv[1], xv[2], xv[3]};
        if (EPL == 8) *(float4*)(a.x + (size_t)m * a.H + k0 + 4) = float4{xv[4 % EPL], xv[5 % EPL], xv[6 % EPL], xv[7 % EPL]};
        typedef T __attribute__((ext_vector_type(EPL))) tv;
        const tv gv = *(const tv*)(g + k0);
        float ov[EPL];
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
            ss += xv[e] * xv[e];
            ov[e] = xv[e] * to_f32(gv[e]);
        }
        put_operand_run<T>((T*)a.op_hi, (T*)a.op_lo, xfrag_elem<T>(m, k0, a.MT), ov, a.op_f16 != 0);
    }
    __shared__ float s_ss[8];
    ss = wave_sum(ss);
    if (threadIdx.x % WAVE == 0) s_ss[threadIdx.x / WAVE] = ss;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int w = 0; w < (int)(blockDim.x / WAVE); ++w) t += s_ss[w];
        a.sq[m] = t;
    }
}

// ---------------------------------------------------------------------------
// Fused skinny weight-streaming GEMM
//
//   Y[m][n] = r_m * ( sum_k W[n][k] X[m][k]  +  s * sum_j B[n][j] u[m][j] ),
//   u[m][j] = sum_k A[j][k] X[m][k]                    (LoRA, adapter on)
//
// which is the LoRA-adapted projection of the normalised row r_m * X[m] (the
// RMSNorm gain is already inside X; r_m is 1/rms of row m from the producer's
// sum-of-squares partials, 1 when n_sq = 0).
//
// A work-group owns one 16-row tile of W (and, with split-K, one of `ksplit`
// slices of K); its NW waves take the tile's fragments round-robin, so every
// weight fragment is read once, as one contiguous 1 KiB wavefront load, and
// feeds MG m-tiles of MFMA (twice when the operand is carried as bf16 value +
// residual).  Each batch of loads (W, X and the LoRA A fragments) is issued
// before its MFMAs.  The LoRA shrink runs on the same operand fragments; each
// wave applies the expand to its own partial u (16x16x16 MFMA, u as bf16
// value + residual) before the single cross-wave reduction, which is valid
// because the expand is linear.  With split-K the slices write partial tiles;
// the last slice to arrive (device-scope counter) sums them in slice order and
// runs the epilogue.
// ---------------------------------------------------------------------------
template <int EPI> struct FG {
    // waves per work-group
    static constexpr int NW = (EPI == EPI_ARGMAX || EPI == EPI_SWIGLU) ? 4 : 8;
    static constexpr int NSRC = (EPI == EPI_SWIGLU) ? 2 : 1;      // LoRA shrink sources
    // work-groups per CU the register budget must allow (SwiGLU: 384+ tiles on 256 CUs)
    static constexpr int MINB = (EPI == EPI_SWIGLU) ? 2 : 1;
    // fragments per wave and load batch: about 112 VGPRs of loads in flight,
    // less what the shrink partials of ranks above 16 take (the work-group
    // runs two waves per SIMD: 256 VGPRs per lane in all)
    template <typename T, int MG, bool SPLIT, int LRT>
    static constexpr int unroll() {
        constexpr int per = 4 + 4 * MG * (SPLIT ? 2 : 1) + 4 * NSRC * LRT;
        constexpr int extra = LRT > 1 ? 12 * NSRC * (LRT - 1) * MG + 8 * (LRT - 1)
                            : (LRT == 1 && sizeof(T) == 4) ? 8 * NSRC * MG + (EPI == EPI_RESID ? 16 : 0) : 0;
        constexpr int budget = 112 - extra > 24 ? 112 - extra : 24;
        constexpr int u = budget / per;
        return u < 1 ? 1 : (u > 6 ? 6 : u);
    }
    // largest m-group the shrink accumulators allow: NSRC * LRT * MG <= 8
    // (32 VGPRs of shrink partials per lane)
    static constexpr int mg_cap(int lrt) {
        return lrt == 0 ? 8 : (8 / (NSRC * lrt) >= 4 ? 4 : 8 / (NSRC * lrt) >= 2 ? 2 : 1);
    }
};

// acc += A(4 k per lane) * p, with p carried as bf16 value + bf16 residual
__device__ __forceinline__ void mma_k4_split(f32x4& acc, const uint2& a, const f32x4& p) {
    f32x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        h[e] = (float)(bf16)p[e];
        l[e] = p[e] - h[e];
    }
    mma_k4(acc, a, h);
    mma_k4(acc, a, l);
}
__device__ __forceinline__ void mma_k4_split(f32x4& acc, const uint4& a, const f32x4& p) { mma_k4(acc, a, p); }

template <typename T, int EPI, int MG, bool SPLIT, int LRT>
__global__ __launch_bounds__(FG<EPI>::NW * 64, FG<EPI>::MINB) void k_fgemm(FGemmArgs a) {
    constexpr int NW = FG<EPI>::NW;
    constexpr int NSRC = FG<EPI>::NSRC;
    constexpr int UNR = FG<EPI>::template unroll<T, MG, SPLIT, LRT>();
    constexpr int NROW = MG * 16;
    typedef typename K4<T>::raw braw;
    __shared__ f32x4 s_red[NW][MG][WAVE];
    __shared__ float s_tile[MG][16][17];
    __shared__ float s_rm[NROW];
    __shared__ float s_sq[NW * 64];
    __shared__ int s_last;

    const int lane = threadIdx.x % WAVE;
    const int wid = threadIdx.x / WAVE;
    const int lrow = lane % 16, lgrp = lane / 16;
    const int S = a.ksplit;
    const int tile = blockIdx.x % a.n_tiles;
    const int ks = blockIdx.x / a.n_tiles;
    const int kb = a.kb;
    const int kbs = ceil_div(kb, S);
    const int f_lo = ks * kbs, f_hi = min(kb, f_lo + kbs);
    const uint4* wt = a.w + (size_t)tile * kb * WAVE;
    const uint4* la[NSRC];
    la[0] = a.la[0];
    if (NSRC > 1) la[NSRC - 1] = a.la[1];
    if (a.lora_mode == LORA_BY_TILE)
        la[0] = tile < a.tile_split0 ? a.la[0] : (tile < a.tile_split1 ? a.la[1] : a.la[2]);
    // LoRA expand blocks of this tile (lane: row lrow, r = 16 t + 4 lgrp + e),
    // scaled by s; for SwiGLU tiles rows 0-7 take source 0 (gate), 8-15 source 1 (up)
    braw bv[LRT > 0 ? LRT : 1];

    for (int mg0 = 0; mg0 < a.MT; mg0 += MG) {
        const int mgn = min(MG, a.MT - mg0);
        f32x4 acc[MG];
        f32x4 uacc[NSRC][LRT > 0 ? LRT * MG : 1];
#pragma unroll
        for (int i = 0; i < MG; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int sc = 0; sc < NSRC; ++sc)
#pragma unroll
            for (int i = 0; i < LRT * MG; ++i) uacc[sc][i] = f32x4{0.f, 0.f, 0.f, 0.f};

        // one batch of fragment loads: W, the operand (value and residual) and
        // the LoRA A fragments of fragments base + NW*u
        uint4 wv[UNR];
        uint4 xh[UNR][MG];
        uint4 xl[UNR][MG];
        uint4 av[UNR][NSRC][LRT > 0 ? LRT : 1];
        auto issue = [&](int base) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int f = base + NW * u;
                const bool fl = f < f_hi;
                const int fc = fl ? f : f_lo;               // always a valid fragment
                wv[u] = wt[(size_t)fc * WAVE + lane];
#pragma unroll
                for (int mt = 0; mt < MG; ++mt) {
                    xh[u][mt] = uint4{0, 0, 0, 0};
                    xl[u][mt] = uint4{0, 0, 0, 0};
                    if (fl && mt < mgn && (mg0 + mt) * 16 + lrow < a.M) {
                        const size_t xi = ((size_t)f * a.MT + mg0 + mt) * WAVE + lane;
                        xh[u][mt] = a.xhi[xi];
                        if (SPLIT) xl[u][mt] = a.xlo[xi];
                    }
                }
#pragma unroll
                for (int sc = 0; sc < NSRC; ++sc)
#pragma unroll
                    for (int t = 0; t < LRT; ++t) av[u][sc][t] = la[sc][((size_t)t * kb + fc) * WAVE + lane];
            }
        };
        auto compute = [&](int base) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                if (base + NW * u >= f_hi) continue;
#pragma unroll
                for (int mt = 0; mt < MG; ++mt) {
                    mma_frag<T>(acc[mt], wv[u], xh[u][mt]);
                    if (SPLIT) mma_frag<T>(acc[mt], wv[u], xl[u][mt]);
                }
#pragma unroll
                for (int sc = 0; sc < NSRC; ++sc)
#pragma unroll
                    for (int t = 0; t < LRT; ++t)
#pragma unroll
                        for (int mt = 0; mt < MG; ++mt) {
                            mma_frag<T>(uacc[sc][t * MG + mt], av[u][sc][t], xh[u][mt]);
                            if (SPLIT) mma_frag<T>(uacc[sc][t * MG + mt], av[u][sc][t], xl[u][mt]);
                        }
            }
        };
        int base = f_lo + wid;
        if (base < f_hi) issue(base);
#pragma unroll
        for (int t = 0; t < LRT; ++t)
            __builtin_memcpy(&bv[t], (const T*)a.lb + (((size_t)tile * LRT + t) * WAVE + lane) * 4, sizeof(braw));
        // LoRA scale per m-tile (0 for rows without the adapter: the lane's u
        // column is block row lrow of the m-tile), formed while the loads fly
        float lsc[MG];
#pragma unroll
        for (int mt = 0; mt < MG; ++mt) {
            lsc[mt] = a.scale;
            if (LRT > 0 && a.adapter_from > 0 && ((mg0 + mt) * 16 + lrow) % a.W < a.adapter_from) lsc[mt] = 0.f;
        }

        // requested after the first weight batch so that they do not delay it:
        // row sums of squares for r_m (thread: row sq_row, partials sq_slice +
        // NSLICE*i), the residual epilogue's x slice and next-norm gains
        constexpr int NSLICE = NW * 64 / NROW;
        constexpr int SQN = 8;
        const int sq_row = threadIdx.x % NROW, sq_slice = threadIdx.x / NROW;
        const int sq_m = mg0 * 16 + sq_row;
        const bool sq_live = a.n_sq > 0 && sq_m < a.M;
        float sqv[SQN];
        if (a.n_sq > 0) {
            // unconditional loads from clamped, valid indices; masked when summed
            const int mc = min(sq_m, a.M - 1);
#pragma unroll
            for (int i = 0; i < SQN; ++i) sqv[i] = a.sq[(size_t)min(sq_slice + NSLICE * i, a.n_sq - 1) * a.sq_stride + mc];
        }
        float4 xr[4];
        typedef T __attribute__((ext_vector_type(16))) t16;
        t16 gq;
        const int em = mg0 * 16 + threadIdx.x;
        const bool e_live = EPI == EPI_RESID && threadIdx.x < mgn * 16 && em < a.M;
        if (e_live) {
            const float4* xs = (const float4*)(a.x + (size_t)em * a.ldx + tile * 16);
#pragma unroll
            for (int i = 0; i < 4; ++i) xr[i] = xs[i];
            gq = *(const t16*)((const T*)a.gnext + tile * 16);
        }

        while (base < f_hi) {
            compute(base);
            base += NW * UNR;
            if (base < f_hi) issue(base);
        }
        float sq_part = 0.f;
        if (sq_live) {
#pragma unroll
            for (int i = 0; i < SQN; ++i)
                if (sq_slice + NSLICE * i < a.n_sq) sq_part += sqv[i];
        }
        if (sq_live)
            for (int pidx = sq_slice + NSLICE * SQN; pidx < a.n_sq; pidx += NSLICE)
                sq_part += a.sq[(size_t)pidx * a.sq_stride + sq_m];

        // this wave's LoRA expand: acc += s * B u_wave
#pragma unroll
        for (int sc = 0; sc < NSRC; ++sc)
#pragma unroll
            for (int t = 0; t < LRT; ++t) {
                braw b = bv[t];
                if (EPI == EPI_SWIGLU && ((lrow < 8) != (sc == 0))) b = braw{};
#pragma unroll
                for (int mt = 0; mt < MG; ++mt) mma_k4_split(acc[mt], b, uacc[sc][t * MG + mt] * lsc[mt]);
            }

        // finish r_m = rsqrt(mean(x^2) + eps) (fixed summation order)
        s_sq[threadIdx.x] = sq_part;
#pragma unroll
        for (int mt = 0; mt < MG; ++mt) s_red[wid][mt][lane] = acc[mt];
        lds_sync();
        if (threadIdx.x < NROW) {
            float sm = 0.f;
            for (int sl = 0; sl < NSLICE; ++sl) sm += s_sq[sl * NROW + threadIdx.x];
            s_rm[threadIdx.x] = a.n_sq > 0 ? rsqrtf(sm / (float)a.norm_dim + a.eps) : 1.f;
        }
        // cross-wave reduction of the tile (fixed order)
        for (int idx = threadIdx.x; idx < MG * WAVE * 4; idx += blockDim.x) {
            const int mt = idx / (WAVE * 4), ln = (idx / 4) % WAVE, e = idx % 4;
            float v = 0.f;
#pragma unroll
            for (int w = 0; w < NW; ++w) v += s_red[w][mt][ln][e];
            s_tile[mt][(ln / 16) * 4 + e][ln % 16] = v;
        }
        lds_sync();

        if (S > 1) {
            // split-K: publish this slice's tile with device-scope (L2-coherent
            // across XCDs) atomic stores, wait for their completion, then count
            // the arrival; the last slice reads the partials with system-scope
            // loads (past any stale L2 line), sums them in slice order and
            // continues with the epilogue.  No cache write-back is needed.
            float* pp = a.part + (size_t)tile * S * (MG * 256);
            for (int idx = threadIdx.x; idx < MG * 256; idx += blockDim.x) {
                const int mt = idx / 256, n = (idx / 16) % 16, ml = idx % 16;
                __hip_atomic_store(pp + (size_t)ks * (MG * 256) + idx, s_tile[mt][n][ml], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            lds_sync();
            if (threadIdx.x == 0)
                s_last = __hip_atomic_fetch_add(a.cnt + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                         (unsigned)(S - 1);
            lds_sync();
            if (!s_last) return;
            for (int idx = threadIdx.x; idx < MG * 256; idx += blockDim.x) {
                const int mt = idx / 256, n = (idx / 16) % 16, ml = idx % 16;
                float pv[KSPLIT_MAX];
#pragma unroll
                for (int k2 = 0; k2 < KSPLIT_MAX; ++k2)
                    pv[k2] = k2 < S ? __hip_atomic_load(pp + (size_t)k2 * (MG * 256) + idx, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_SYSTEM)
                                    : 0.f;
                float v = 0.f;
#pragma unroll
                for (int k2 = 0; k2 < KSPLIT_MAX; ++k2) v += pv[k2];
                s_tile[mt][n][ml] = v;
            }
            if (threadIdx.x == 0) __hip_atomic_store(a.cnt + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            lds_sync();
        }

        // epilogues (r_m applied here)
        if (EPI == EPI_STORE) {
            for (int idx = threadIdx.x; idx < mgn * 256; idx += blockDim.x) {
                const int mt = idx / 256, n = idx % 16, ml = (idx / 16) % 16;
                const int m = (mg0 + mt) * 16 + ml;
                if (m < a.M) a.out[(size_t)m * a.ldo + tile * 16 + n] = s_tile[mt][n][ml] * s_rm[mt * 16 + ml];
            }
        } else if (EPI == EPI_RESID) {
            // x += tile; next operand x * g_next; per-row sum of squares over the 16 columns
            if (e_live) {
                const int mt = threadIdx.x / 16, ml = threadIdx.x % 16;
                const int m = em;
                const float rm = s_rm[threadIdx.x];
                float ss = 0.f;
                float xv[16];
#pragma unroll
                for (int n = 0; n < 16; ++n) {
                    xv[n] = xr[n / 4][n % 4] + s_tile[mt][n][ml] * rm;
                    ss += xv[n] * xv[n];
                }
                float4* xd = (float4*)(a.x + (size_t)m * a.ldx + tile * 16);
#pragma unroll
                for (int i = 0; i < 4; ++i) xd[i] = float4{xv[4 * i], xv[4 * i + 1], xv[4 * i + 2], xv[4 * i + 3]};
                constexpr int EPL = Elt<T>::EPL;
#pragma unroll
                for (int n0 = 0; n0 < 16; n0 += EPL) {
                    float ov[EPL];
#pragma unroll
                    for (int i = 0; i < EPL; ++i) ov[i] = xv[n0 + i] * to_f32(gq[n0 + i]);
                    put_operand_run<T>((T*)a.nx_hi, (T*)a.nx_lo, xfrag_elem<T>(m, tile * 16 + n0, a.n_MT), ov);
                }
                a.sq_out[(size_t)tile * a.sq_stride + m] = ss;
            }
        } else if (EPI == EPI_SWIGLU) {
            // tile rows 0-7: gate rows 8*tile..; rows 8-15: the matching up rows;
            // a thread writes one run of EPL consecutive h columns of one row
            constexpr int EPL = Elt<T>::EPL;
            constexpr int RUNS = 8 / EPL;
            for (int idx = threadIdx.x; idx < mgn * 16 * RUNS; idx += blockDim.x) {
                const int mt = idx / (16 * RUNS), ml = (idx / RUNS) % 16, c0 = (idx % RUNS) * EPL;
                const int m = (mg0 + mt) * 16 + ml;
                if (m < a.M) {
                    const float rm = s_rm[mt * 16 + ml];
                    float hv[EPL];
#pragma unroll
                    for (int i = 0; i < EPL; ++i) {
                        const float gt = s_tile[mt][c0 + i][ml] * rm;
                        const float up = s_tile[mt][c0 + i + 8][ml] * rm;
                        hv[i] = gt / (1.f + __expf(-gt)) * up;
                    }
                    put_operand_run<T>((T*)a.nx_hi, (T*)a.nx_lo, xfrag_elem<T>(m, tile * 8 + c0, a.n_MT), hv);
                }
            }
        } else {  // EPI_ARGMAX: tied LM head, per-tile (max, argmax) per row
            for (int idx = threadIdx.x; idx < mgn * 16; idx += blockDim.x) {
                const int mt = idx / 16, ml = idx % 16;
                const int m = (mg0 + mt) * 16 + ml;
                if (m >= a.M) continue;
                const float rm = s_rm[idx];
                float best = -INFINITY;
                int bi = 0x7fffffff;
                const int excl = m % a.W >= a.excl_from ? a.exclude : -1;
                for (int n = 0; n < 16; ++n) {
                    const int v = tile * 16 + n;
                    const float val = s_tile[mt][n][ml] * rm;
                    if (a.logits) a.logits[(size_t)m * a.ldo + v] = val;
                    if (v == excl) continue;
                    if (val > best) { best = val; bi = v; }   // ascending v: first max wins ties
                }
                a.arg_val[(size_t)tile * a.M + m] = best;
                a.arg_idx[(size_t)tile * a.M + m] = bi;
                if (a.arg_sum) {     // softmax partial over all 16 columns
                    float mx = -INFINITY;
                    for (int n = 0; n < 16; ++n) mx = fmaxf(mx, s_tile[mt][n][ml] * rm);
                    float sm = 0.f;
                    if (mx > -INFINITY)
                        for (int n = 0; n < 16; ++n) sm += expf(s_tile[mt][n][ml] * rm - mx);
                    a.arg_mx[(size_t)tile * a.M + m] = mx;
                    a.arg_sum[(size_t)tile * a.M + m] = sm;
                }
            }
        }
        lds_sync();
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
// O^T += V^T P^T takes P^T directly from the score accumulators.  The four
// waves take key blocks round-robin and merge in LDS at the end.
// ---------------------------------------------------------------------------

// Prefill chunk: per-head RMSNorm and RoPE of the chunk's keys, appended to
// the cache with the values before the chunk's attention reads them.  One
// work-group per (16 rows, KV head, sequence); 16 lanes per row.
template <typename T, int HD>
__global__ __launch_bounds__(256) void k_kvwrite(KVWriteArgs a) {
    typedef RowPrep<T, HD> RP;
    constexpr int NP = RP::NP, HALF = RP::HALF;
    __shared__ T s_row[16][HD];
    const int g = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    const int lrow = lane % 16, lgrp = lane / 16;
    const int r = 4 * wid + lgrp;
    const int j = blockIdx.x * 16 + r;
    const int t = a.pos0[b], nrows = a.nrows[b];
    const bool live = j < a.W && j < nrows;
    const int jj = live ? j : 0;                        // dead rows read a valid row
    const float* ks = a.qkv + ((size_t)b * a.W + jj) * a.nqkv + (size_t)a.n_q * HD + (size_t)g * HD;
    const float* vs = ks + (size_t)a.n_kv * HD;
    RP rk;
    rk.load(ks, a.rope + (size_t)(t + jj) * HALF, lrow);
    const typename RP::fv vlo = *(const typename RP::fv*)(vs + NP * lrow);
    const typename RP::fv vhi = *(const typename RP::fv*)(vs + HALF + NP * lrow);
    Gains<T, HD> gk;
    if (a.qk_norm) gk.load(a.k_norm, lrow);
    float g_lo[NP], g_hi[NP];
    gk.get(a.qk_norm, g_lo, g_hi);
    T klo[NP], khi[NP];
    rk.finish(s_row[r], live, g_lo, g_hi, a.qk_norm, a.eps, lrow, klo, khi);
    if (!live) return;
    const int pos = t + j;
    const size_t head = (((size_t)a.layer * a.max_batch + b) * a.n_kv + g) * a.nblk * 16 * HD;
    T* kblk = (T*)a.kcache + head + (size_t)(pos / 16) * 16 * HD;
    T* vblk = (T*)a.vcache + head + (size_t)(pos / 16) * 16 * HD;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const int i0 = NP * lrow + p;
        kblk[kblock_elem<T>(pos % 16, i0)] = klo[p];
        kblk[kblock_elem<T>(pos % 16, i0 + HALF)] = khi[p];
        vblk[vblock_elem(pos % 16, i0)] = from_f32<T>(vlo[p]);
        vblk[vblock_elem(pos % 16, i0 + HALF)] = from_f32<T>(vhi[p]);
    }
}

constexpr float RESCALE_SLACK = 8.f;

template <typename T, int HD, int QT>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
    constexpr int FK = Elt<T>::FK;
    constexpr int EPL = Elt<T>::EPL;
    constexpr int NDS = HD / FK;          // fragments per key row
    constexpr int NDT = HD / 16;          // V^T tiles
    constexpr int QROWS = QT * 16;
    constexpr int LDQ = HD + 16 / (int)sizeof(T);   // padded LDS row (bank spread)
    constexpr int KBMAX = 48;                       // block keys: W <= 33 -> 3 blocks
    constexpr int LDO = HD + 4;                     // merge rows (16-byte aligned, banks spread)
    constexpr int HALF = HD / 2;
    typedef typename K4<T>::raw vraw;
    typedef RowPrep<T, HD> RP;

    if ((int)blockIdx.x >= a.s_launch) {
        // work-groups past the splits warm the memory-side cache with what
        // the next kernels read (the attention keeps few CUs busy): one word
        // per 128-byte line of this work-group's share of the three ranges
        const int n_pf = (gridDim.x - a.s_launch) * gridDim.y * gridDim.z;
        const int ip = ((blockIdx.x - a.s_launch) * gridDim.y + blockIdx.y) * gridDim.z + blockIdx.z;
        const size_t n0 = a.pf_bytes[0] / 128, n1 = a.pf_bytes[1] / 128, n2 = a.pf_bytes[2] / 128;
        const size_t lines = n0 + n1 + n2;
        const size_t per = (lines + n_pf - 1) / n_pf;
        const size_t l0 = (size_t)ip * per, l1 = min(l0 + per, lines);
        constexpr int PFN = 16;
        unsigned v[PFN];
#pragma unroll
        for (int i = 0; i < PFN; ++i) {
            const size_t li = l0 + (size_t)i * blockDim.x + threadIdx.x;
            const char* p = li < n0 ? a.pf[0] + li * 128
                          : li < n0 + n1 ? a.pf[1] + (li - n0) * 128 : a.pf[2] + (li - n0 - n1) * 128;
            v[i] = li < l1 ? *(const unsigned*)p : 0u;
        }
        unsigned acc = 0;
#pragma unroll
        for (int i = 0; i < PFN; ++i) acc ^= v[i];
        asm volatile("" ::"v"(acc));
        return;
    }
    if (a.skip_prefix) return;                         // every split run by k_attn_rows
    const int s = blockIdx.x, g = blockIdx.y;
    const int b = blockIdx.z / a.n_qgrp;
    const int q0 = (blockIdx.z % a.n_qgrp) * QROWS;      // first query row of this work-group
    const int t = a.pos0[b];
    const int nrows = a.nrows[b];
    // chunk mode (prefill): the chunk's keys are already in the cache; splits
    // s < s_pre cover keys [0, t + nrows) and there is no block split
    const int T_keys = a.chunk ? t + nrows : t;
    int s_pre, chunk;
    attn_splits(T_keys, a.kps, a.chunk ? a.s_launch + 1 : a.s_launch, s_pre, chunk);
    const int W = a.W, G = a.G;
    const int QR = G * W;
    if (a.chunk ? s >= s_pre : s > s_pre) {
        // unused split: mark its partials empty (max -inf, sum 0), so that the
        // merge can read every split without the sequence's position
        const int q = q0 + (int)threadIdx.x;
        if ((int)threadIdx.x < QROWS && q < QR) {
            const size_t pr = (((size_t)b * a.n_q + g * G + q / W) * W + q % W) * a.s_launch + s;
            a.part_ml[pr * 2 + 0] = -INFINITY;
            a.part_ml[pr * 2 + 1] = 0.f;
        }
        return;
    }
    const bool blk = !a.chunk && s == s_pre;             // the split of the W block keys
    const int k_lo = blk ? t : min(s * chunk, T_keys);
    const int k_hi = blk ? t : min(T_keys, k_lo + chunk);

    extern __shared__ __align__(16) unsigned char smem[];
    T* q_l = (T*)smem;                                   // [QROWS][LDQ]
    T* kb_l = q_l + QROWS * LDQ;                         // [KBMAX][LDQ]
    T* vb_l = kb_l + KBMAX * LDQ;                        // [KBMAX][HD]
    float* obuf = (float*)smem;                          // [2][QROWS][LDO], aliases after the key loop
    float* ml_l = (float*)(smem + a.smem_main);          // [4][QROWS][2]

    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    const int lrow = lane % 16, lgrp = lane / 16;
    const size_t row_stride = (size_t)a.nqkv;
    const float* qkv_b = a.qkv + (size_t)b * W * row_stride;
    const float2* rope = a.rope;

    T* kc = (T*)a.kcache + (((size_t)a.layer * a.max_batch + b) * a.n_kv + g) * a.nblk * 16 * HD;
    T* vc = (T*)a.vcache + (((size_t)a.layer * a.max_batch + b) * a.n_kv + g) * a.nblk * 16 * HD;
    const int kb_first = k_lo / 16;
    const int n_pref = (k_hi > k_lo) ? ceil_div(k_hi, 16) - kb_first : 0;
    const int nkb_blk = blk ? ceil_div(W, 16) : 0;
    const int n_items = n_pref + nkb_blk;

    // item it < n_pref: prefix key block kb_first + it from the cache;
    // otherwise block keys 16*(it - n_pref) .. from LDS
    auto load_item = [&](int it, uint4* kf, vraw* vf) {
        if (it < n_pref) {
            const T* kblk = kc + (size_t)(kb_first + it) * 16 * HD;
            const T* vblk = vc + (size_t)(kb_first + it) * 16 * HD;
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds) kf[ds] = *(const uint4*)(kblk + (size_t)(ds * WAVE + lane) * EPL);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) vf[dt] = *(const vraw*)(vblk + (size_t)(dt * WAVE + lane) * 4);
        } else {
            const int bb = it - n_pref;
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
    };

    // A wave takes key blocks it, it+4, ... in chunks of CH blocks: the scores
    // of a chunk are formed first, so the running max and the rescale of the
    // accumulated output happen once per chunk (not at all for the first one).
    // The wave's first chunk of prefix blocks is requested before the query
    // preparation, which it does not depend on.  Splits of cache keys hold two
    // chunks in registers (the next one loading), so CH is the largest of
    // 4, 2, 1 for which those, the output accumulators and the Q fragments
    // fit a budget of 304 registers per lane (beyond it the compiler spills).
    // A single query tile takes one block per chunk: the work-group then fits
    // in 256 registers per lane, two waves per SIMD, which hides more of the
    // chain than larger chunks do (measured on the batch-1 step).
    // With four or more query tiles the Q fragments are read from LDS at each
    // use instead of being held in registers.
    constexpr bool QF_LDS = QT >= 4;
    constexpr int R_BLK = NDS * 4 + NDT * (int)(sizeof(vraw) / 4);    // one key block's K and V
    constexpr int R_FIX = QT * (NDT * 4 + (QF_LDS ? 0 : NDS * 4));
    constexpr int CH = (QT == 1 || QF_LDS) ? 1 : 8 * R_BLK + R_FIX <= 304 ? 4 : 4 * R_BLK + R_FIX <= 304 ? 2 : 1;
    uint4 kn[CH][NDS];
    vraw vn[CH][NDT];
    auto load_chunk = [&](int it0) {
#pragma unroll
        for (int c = 0; c < CH; ++c)
            if (it0 + 4 * c < n_items) load_item(it0 + 4 * c, kn[c], vn[c]);
    };
    // prefix block it from the cache (it clamped into range by the caller)
    auto load_pref = [&](int it, uint4* kf, vraw* vf) {
        const T* kblk = kc + (size_t)(kb_first + it) * 16 * HD;
        const T* vblk = vc + (size_t)(kb_first + it) * 16 * HD;
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds) kf[ds] = *(const uint4*)(kblk + (size_t)(ds * WAVE + lane) * EPL);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) vf[dt] = *(const vraw*)(vblk + (size_t)(dt * WAVE + lane) * 4);
    };
    // splits of prefix keys only: every load is unconditional (indexes past the
    // wave's last block repeat that block), so that the compiler's wait before
    // a chunk's products covers that chunk's loads and not the next chunk's
    const bool pipe = !blk && n_items > 0;
    if (pipe) {
#pragma unroll
        for (int c = 0; c < CH; ++c) load_pref(min(wid + 4 * c, n_items - 1), kn[c], vn[c]);
    } else if (!blk) {
        load_chunk(wid);
    }

    // -- Q rows (and, in the block split, K/V rows): all loads first, then
    //    norm + rotation; wave w, lane group lgrp handles rows 16*i + 4*w + lgrp
    constexpr int QSTEPS = QROWS / 16;
    constexpr int KSTEPS = KBMAX / 16;
    Gains<T, HD> gq;
    if (a.qk_norm) gq.load(a.q_norm, lrow);
    RP rp[QSTEPS];
#pragma unroll
    for (int i = 0; i < QSTEPS; ++i) {
        const int q = q0 + 16 * i + 4 * wid + lgrp;
        const int qq = (q < QR && (q % W) < nrows) ? q : 0;   // dead rows read a valid row
        rp[i].load(qkv_b + (size_t)(qq % W) * row_stride + (size_t)(g * G + qq / W) * HD,
                   rope + (size_t)(t + qq % W) * HALF, lrow);
    }
    float gq_lo[RP::NP], gq_hi[RP::NP];
    // the softmax scale (log2 e / sqrt(head_dim)) rides on the query gains:
    // the rotation is linear, so the scores come out of the MFMA scaled
    auto scale_gains = [&](float* lo_, float* hi_) {
#pragma unroll
        for (int p = 0; p < RP::NP; ++p) {
            lo_[p] *= a.scale_log2;
            hi_[p] *= a.scale_log2;
        }
    };
    if (blk) {
        Gains<T, HD> gk;
        if (a.qk_norm) gk.load(a.k_norm, lrow);
        RP rk[KSTEPS];
        typename RP::fv vlo[KSTEPS], vhi[KSTEPS];
#pragma unroll
        for (int i = 0; i < KSTEPS; ++i) {
            const int j = 16 * i + 4 * wid + lgrp;
            const int jj = (j < W && j < nrows) ? j : 0;
            const float* ks = qkv_b + (size_t)jj * row_stride + (size_t)a.n_q * HD + (size_t)g * HD;
            const float* vs = ks + (size_t)a.n_kv * HD;
            rk[i].load(ks, rope + (size_t)(t + jj) * HALF, lrow);
            vlo[i] = *(const typename RP::fv*)(vs + RP::NP * lrow);
            vhi[i] = *(const typename RP::fv*)(vs + HALF + RP::NP * lrow);
        }
        gq.get(a.qk_norm, gq_lo, gq_hi);
        scale_gains(gq_lo, gq_hi);
#pragma unroll
        for (int i = 0; i < QSTEPS; ++i) {
            const int ql = 16 * i + 4 * wid + lgrp;
            T lo[RP::NP], hi[RP::NP];
            rp[i].finish(q_l + ql * LDQ, q0 + ql < QR, gq_lo, gq_hi, a.qk_norm, a.eps, lrow, lo, hi);
        }
        // block keys and values; the verify appends them to the cache
        float gk_lo[RP::NP], gk_hi[RP::NP];
        gk.get(a.qk_norm, gk_lo, gk_hi);
#pragma unroll
        for (int i = 0; i < KSTEPS; ++i) {
            const int j = 16 * i + 4 * wid + lgrp;
            if (j >= nkb_blk * 16) continue;
            const bool live = j < W && j < nrows;
            T klo[RP::NP], khi[RP::NP], vl[RP::NP], vh[RP::NP];
            rk[i].finish(kb_l + j * LDQ, live, gk_lo, gk_hi, a.qk_norm, a.eps, lrow, klo, khi);
            T* vd = vb_l + j * HD;
#pragma unroll
            for (int p = 0; p < RP::NP; ++p) {
                vl[p] = from_f32<T>(live ? vlo[i][p] : 0.f);
                vh[p] = from_f32<T>(live ? vhi[i][p] : 0.f);
                vd[RP::NP * lrow + p] = vl[p];
                vd[HALF + RP::NP * lrow + p] = vh[p];
            }
            if (live && j < a.kv_rows && q0 == 0) {
                const int pos = t + j;
                T* kblk = kc + (size_t)(pos / 16) * 16 * HD;
                T* vblk = vc + (size_t)(pos / 16) * 16 * HD;
#pragma unroll
                for (int p = 0; p < RP::NP; ++p) {
                    const int i0 = RP::NP * lrow + p;
                    kblk[kblock_elem<T>(pos % 16, i0)] = klo[p];
                    kblk[kblock_elem<T>(pos % 16, i0 + HALF)] = khi[p];
                    vblk[vblock_elem(pos % 16, i0)] = vl[p];
                    vblk[vblock_elem(pos % 16, i0 + HALF)] = vh[p];
                }
            }
        }
    } else {
        gq.get(a.qk_norm, gq_lo, gq_hi);
        scale_gains(gq_lo, gq_hi);
#pragma unroll
        for (int i = 0; i < QSTEPS; ++i) {
            const int ql = 16 * i + 4 * wid + lgrp;
            T lo[RP::NP], hi[RP::NP];
            rp[i].finish(q_l + ql * LDQ, q0 + ql < QR, gq_lo, gq_hi, a.qk_norm, a.eps, lrow, lo, hi);
        }
    }
    lds_sync();

    // -- Q^T fragments in registers (or read from LDS at each use, QF_LDS)
    uint4 qf[QF_LDS ? 1 : QT][NDS];
    if (!QF_LDS) {
#pragma unroll
        for (int qt = 0; qt < (QF_LDS ? 1 : QT); ++qt)
#pragma unroll
            for (int ds = 0; ds < NDS; ++ds)
                qf[qt][ds] = *(const uint4*)(q_l + (qt * 16 + lrow) * LDQ + ds * FK + lgrp * EPL);
    }
    // z0: a zero the compiler cannot see through, so that the LDS reads stay
    // inside the key loop instead of being hoisted into registers
    auto qfrag = [&](int qt, int ds, int z0) -> uint4 {
        if (QF_LDS) return *(const uint4*)(q_l + z0 + (qt * 16 + lrow) * LDQ + ds * FK + lgrp * EPL);
        return qf[QF_LDS ? 0 : qt][ds];
    };

    // block row of each of this lane's query columns (for the causal mask)
    int jq[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) jq[qt] = (q0 + qt * 16 + lrow) % W;

    f32x4 o_acc[NDT][QT];
    float m_run[QT], l_run[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        m_run[qt] = -1e30f;
        l_run[qt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o_acc[dt][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // One chunk in phases, each straight-line over all query tiles so that
    // the tiles' independent MFMA chains interleave: scores, key masks (only
    // on chunks that reach past the split), one vote on the reference
    // maximum, weights and P.V.
    auto step = [&](int it0, const uint4 (&kcur)[CH][NDS], const vraw (&vcur)[CH][NDT]) {
        const bool first = it0 == wid;
        int z0 = 0;
        if (QF_LDS) asm volatile("s_mov_b32 %0, 0" : "=s"(z0));
        // a chunk whose blocks all lie inside the split's cache keys (below
        // the chunk rows in chunk mode) needs no key mask (wave-uniform)
        bool full = true;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int it = it0 + 4 * c;
            full = full && it < n_items && it < n_pref && (kb_first + it) * 16 + 16 <= (a.chunk ? min(k_hi, t) : k_hi);
        }
        // lane holds keys key0(c) + 4*lgrp + e for query column qt*16 + lrow;
        // masked keys score -inf (weight exp2(-inf) = 0)
        float sv[QT][CH][4];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            f32x4 sc[QT];
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) sc[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (it0 + 4 * c < n_items) {
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
                    for (int qt = 0; qt < QT; ++qt) mma_frag<T>(sc[qt], kcur[c][ds], qfrag(qt, ds, z0));
            }
#pragma unroll
            for (int qt = 0; qt < QT; ++qt)
#pragma unroll
                for (int e = 0; e < 4; ++e) sv[qt][c][e] = sc[qt][e];
        }
        if (!full) {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int it = it0 + 4 * c;
                const bool pref = it < n_pref;
                const int key0 = pref ? (kb_first + it) * 16 : (it - n_pref) * 16;
#pragma unroll
                for (int qt = 0; qt < QT; ++qt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int kk = key0 + lgrp * 4 + e;
                        const bool in_pref = (kk < k_hi) & (!a.chunk | (kk < t) | (kk - t <= jq[qt]));
                        const bool in_blk = (kk < nrows) & ((kk <= jq[qt]) | (jq[qt] >= a.full_from));
                        const bool ok = (it < n_items) & (pref ? in_pref : in_blk);
                        if (!ok) sv[qt][c][e] = -INFINITY;
                    }
            }
        }
        // The reference maximum m_run is set from the wave's first chunk and
        // raised (the output and sum rescaled) only when a score exceeds it by
        // more than RESCALE_SLACK (log2 units, one vote of the wave over all
        // tiles): the weights exp2(s - m_run) stay below 2^RESCALE_SLACK and
        // the ratio of sums is the same for any reference, so only rounding
        // differs.  Otherwise no row maximum is formed.
        bool over = false;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
            for (int c = 0; c < CH; ++c)
#pragma unroll
                for (int e = 0; e < 4; ++e) over = over | (sv[qt][c][e] > m_run[qt] + RESCALE_SLACK);
        if (first || __any(over)) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) {
                float mloc = -1e30f;
#pragma unroll
                for (int c = 0; c < CH; ++c)
#pragma unroll
                    for (int e = 0; e < 4; ++e) mloc = fmaxf(mloc, sv[qt][c][e]);
                const float m_new = fmaxf(m_run[qt], xrow_max(mloc));
                if (!first) {
                    const float corr = __builtin_amdgcn_exp2f(m_run[qt] - m_new);
                    l_run[qt] *= corr;
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) o_acc[dt][qt] *= corr;
                }
                m_run[qt] = m_new;
            }
        }
        // l_run holds this lane's share of the row sum; the four lane groups
        // of a query column are added after the key loop
        f32x4 p[QT][CH];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
            for (int c = 0; c < CH; ++c)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    p[qt][c][e] = __builtin_amdgcn_exp2f(sv[qt][c][e] - m_run[qt]);
                    l_run[qt] += p[qt][c][e];
                }
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            if (it0 + 4 * c >= n_items) continue;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int qt = 0; qt < QT; ++qt) mma_k4(o_acc[dt][qt], vcur[c][dt], p[qt][c]);
        }
    };
    if (pipe) {
        // the next chunk's loads are in flight while the current one is reduced;
        // the last chunk is peeled off so that no load is issued past the end
        uint4 kx[CH][NDS];
        vraw vx[CH][NDT];
        int it0 = wid;
        for (; it0 + 4 * CH < n_items; it0 += 4 * CH) {
#pragma unroll
            for (int c = 0; c < CH; ++c) load_pref(min(it0 + 4 * CH + 4 * c, n_items - 1), kx[c], vx[c]);
            step(it0, kn, vn);
#pragma unroll
            for (int c = 0; c < CH; ++c) {
#pragma unroll
                for (int ds = 0; ds < NDS; ++ds) kn[c][ds] = kx[c][ds];
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) vn[c][dt] = vx[c][dt];
            }
        }
        if (it0 < n_items) step(it0, kn, vn);
    } else {
        if (blk) load_chunk(wid);
        for (int it0 = wid; it0 < n_items; it0 += 4 * CH) {
            step(it0, kn, vn);
            if (it0 + 4 * CH < n_items) load_chunk(it0 + 4 * CH);
        }
    }

#pragma unroll
    for (int qt = 0; qt < QT; ++qt) l_run[qt] = xrow_sum(l_run[qt]);

    // -- merge the four waves: common max per query row, then a two-round tree
    //    (waves 2,3 -> 0,1, then 1 -> 0) in LDS; wave 0 writes the partial
    lds_sync();                                     // LDS operands dead: obuf may alias
    if (lgrp == 0) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
            ml_l[(wid * QROWS + qt * 16 + lrow) * 2 + 0] = m_run[qt];
            ml_l[(wid * QROWS + qt * 16 + lrow) * 2 + 1] = l_run[qt];
        }
    }
    lds_sync();
    float mx[QT];
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int q = qt * 16 + lrow;
        mx[qt] = -1e30f;
#pragma unroll
        for (int w = 0; w < 4; ++w) mx[qt] = fmaxf(mx[qt], ml_l[(w * QROWS + q) * 2]);
        const float f = exp2f(m_run[qt] - mx[qt]);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) o_acc[dt][qt] *= f;
    }
    auto put = [&](float* reg) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                *(f32x4*)(reg + (qt * 16 + lrow) * LDO + dt * 16 + lgrp * 4) = o_acc[dt][qt];
    };
    auto add = [&](const float* reg) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
                o_acc[dt][qt] += *(const f32x4*)(reg + (qt * 16 + lrow) * LDO + dt * 16 + lgrp * 4);
    };
    if (wid >= 2) put(obuf + (wid - 2) * QROWS * LDO);
    lds_sync();
    if (wid < 2) add(obuf + wid * QROWS * LDO);
    lds_sync();
    if (wid == 1) put(obuf);
    lds_sync();
    if (wid != 0) return;
    add(obuf);

    // partial of this split: max (log2 domain), sum, unnormalised output per query row
    const int S = a.s_launch;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
        const int ql = qt * 16 + lrow, q = q0 + ql;     // local and global query row
        if (q >= QR) continue;
        const int gi = q / W, j = q % W;
        const size_t pr = (((size_t)b * a.n_q + g * G + gi) * W + j) * S + s;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) *(f32x4*)(a.part_o + pr * HD + dt * 16 + lgrp * 4) = o_acc[dt][qt];
        if (lgrp == 0) {
            float L = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w)
                L += ml_l[(w * QROWS + ql) * 2 + 1] * exp2f(ml_l[(w * QROWS + ql) * 2] - mx[qt]);
            a.part_ml[pr * 2 + 0] = mx[qt];
            a.part_ml[pr * 2 + 1] = L;
        }
    }
}

// ---------------------------------------------------------------------------
// Attention partials of draft and verify passes with four or five 16-row
// query tiles per KV head (bf16, head_dim 128): the split-KV schedule, block
// split and partial layout of k_attn, another work split.  k_attn gives each
// wave every query tile and a quarter of the keys: 160 accumulator registers
// per lane, copies between accumulator and vector registers at each key
// block, and a merge of the four waves.  Here wave w owns query tile w over
// every key of the work-group (32 accumulator registers, no merge), and the
// keys go through LDS once per work-group:
//  * prefix splits: the first four waves copy each cache block (16 bytes per
//    lane and chunk, one block ahead in registers) into a double buffer;
//  * the block split: the same waves normalise and rotate the W block rows'
//    keys into LDS blocks of the cache layout (and append them to the cache
//    in the verify), once the query fragments are in registers;
//  * unused splits mark their partials empty.
// Several work-groups share a CU.
// ---------------------------------------------------------------------------

// 16 wait states, with nothing scheduled across: enough for any MFMA of this
// file to finish writing its result, or reading its operands, before the
// instructions that follow touch those registers
__device__ __forceinline__ void mfma_settle() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

constexpr int ATTN_ROWS_WMAX = 48;     // block rows of the block split (three key blocks)

// Four work-groups per CU (16 or 20 waves) need at most 128 or 102
// registers per lane: the waves-per-SIMD floor holds the allocator to that.
template <int QT>
__global__ __launch_bounds__(QT * 64) __attribute__((amdgpu_waves_per_eu(QT, 8))) void k_attn_rows(AttnArgs a) {
    typedef bf16 T;
    constexpr int HD = 128, HALF = HD / 2, FK = Elt<T>::FK, EPL = Elt<T>::EPL;
    constexpr int NDS = HD / FK, NDT = HD / 16;
    constexpr int LDQ = HD + 16 / (int)sizeof(T);
    constexpr int BLK = 2 * 16 * HD * (int)sizeof(T);       // one key block's K then V (8 KiB)
    constexpr int NLD = 4;                                   // waves that stage the blocks
    constexpr int CPL = BLK / 16 / (NLD * WAVE);             // 16-byte chunks per staging lane
    constexpr int Q_BYTES = (QT * 16 * LDQ * (int)sizeof(T) + 15) / 16 * 16;
    typedef uint2 vraw;
    typedef RowPrep<T, HD> RP;
    static_assert(QT >= NLD && CPL * NLD * WAVE * 16 == BLK, "staging layout");
    static_assert((ATTN_ROWS_WMAX / 16) * BLK <= Q_BYTES + 2 * BLK, "block split keys fit the LDS");

    const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int t = a.pos0[b], nrows = a.nrows[b];
    int s_pre, chunk;
    attn_splits(t, a.kps, a.s_launch, s_pre, chunk);
    const int W = a.W, G = a.G, QR = G * W;
    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    const int lrow = lane % 16, lgrp = lane / 16;
    const int q = wid * 16 + lrow;                             // this lane's query column
    if (s > s_pre) {
        // unused split: partials empty (max -inf, sum 0), so that the merge
        // can read every split without the sequence's position
        if (lgrp == 0 && q < QR) {
            const size_t pr = (((size_t)b * a.n_q + g * G + q / W) * W + q % W) * a.s_launch + s;
            a.part_ml[pr * 2 + 0] = -INFINITY;
            a.part_ml[pr * 2 + 1] = 0.f;
        }
        return;
    }
    const bool blk = s == s_pre;                               // the split of the W block keys
    const int k_lo = blk ? t : min(s * chunk, t), k_hi = blk ? t : min(t, k_lo + chunk);
    const int kb_first = k_lo / 16;
    const int n_items = blk ? ceil_div(W, 16) : k_hi > k_lo ? ceil_div(k_hi, 16) - kb_first : 0;

    extern __shared__ __align__(16) unsigned char smem[];
    T* q_l = (T*)smem;                                         // [QT * 16][LDQ]
    unsigned char* kv_l = smem + Q_BYTES;                      // [2][BLK]

    const size_t row_stride = (size_t)a.nqkv;
    const float* qkv_b = a.qkv + (size_t)b * W * row_stride;
    const size_t head = (((size_t)a.layer * a.max_batch + b) * a.n_kv + g) * a.nblk * 16 * HD;
    const unsigned char* kc = (const unsigned char*)((const T*)a.kcache + head);
    const unsigned char* vc = (const unsigned char*)((const T*)a.vcache + head);

    // prefix staging: chunk c of a block is 16 bytes at c * 16 (K: c < BLK /
    // 32, then V); staging lane (wid, lane) holds chunks (wid * CPL + k) *
    // WAVE + lane (two named registers, not an array: an array captured by the
    // staging helpers is placed in scratch memory)
    static_assert(CPL == 2, "two staging chunks per lane");
    auto gchunk = [&](int it, int k) -> uint4 {
        const size_t off = (size_t)(kb_first + it) * (BLK / 2);
        const int c = (wid * CPL + k) * WAVE + lane;
        return c < BLK / 32 ? *(const uint4*)(kc + off + (size_t)c * 16)
                            : *(const uint4*)(vc + off + (size_t)(c - BLK / 32) * 16);
    };
    auto schunk = [&](int buf, int k, const uint4& v) {
        const int c = (wid * CPL + k) * WAVE + lane;
        *(uint4*)(kv_l + (size_t)buf * BLK + (size_t)c * 16) = v;
    };
    uint4 stg0 = uint4{0u, 0u, 0u, 0u}, stg1 = uint4{0u, 0u, 0u, 0u};
    auto gload = [&](int it) { stg0 = gchunk(it, 0); stg1 = gchunk(it, 1); };
    auto swrite = [&](int buf) { schunk(buf, 0, stg0); schunk(buf, 1, stg1); };
    const bool stager = wid < NLD;
    if (stager && !blk && n_items > 0) gload(0);

    // -- this wave's 16 query rows: normed, rotated and scaled by
    //    log2 e / sqrt(head_dim) into LDS, four rows per step, in two halves
    //    (the first key block's loads are in flight meanwhile)
    {
        Gains<T, HD> gq;
        if (a.qk_norm) gq.load(a.q_norm, lrow);
        float gq_lo[RP::NP], gq_hi[RP::NP];
        gq.get(a.qk_norm, gq_lo, gq_hi);
#pragma unroll
        for (int p = 0; p < RP::NP; ++p) {
            gq_lo[p] *= a.scale_log2;
            gq_hi[p] *= a.scale_log2;
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            RP rp[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int qi = wid * 16 + 4 * (2 * h + i) + lgrp;
                const int qq = (qi < QR && (qi % W) < nrows) ? qi : 0;   // dead rows read a valid row
                rp[i].load(qkv_b + (size_t)(qq % W) * row_stride + (size_t)(g * G + qq / W) * HD,
                           a.rope + (size_t)(t + qq % W) * HALF, lrow);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int qi = wid * 16 + 4 * (2 * h + i) + lgrp;
                T lo[RP::NP], hi[RP::NP];
                rp[i].finish(q_l + qi * LDQ, qi < QR, gq_lo, gq_hi, a.qk_norm, a.eps, lrow, lo, hi);
            }
        }
    }
    if (stager && !blk && n_items > 0) {
        swrite(0);
        if (n_items > 1) gload(1);
    }
    lds_sync();
    uint4 qf[NDS];
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds) qf[ds] = *(const uint4*)(q_l + q * LDQ + ds * FK + lgrp * EPL);

    if (blk) {
        // block keys and values into LDS key blocks 0 .. n_items - 1 (over the
        // query rows, read above); row r = 4 wid + lgrp of each block, 16
        // lanes per row.  The verify appends rows j < kv_rows to the cache.
        lds_sync();
        if (stager) {
            static_assert(EPL == 8 && RP::NP == 4, "bf16 block layout with four pairs per lane");
            Gains<T, HD> gk;
            if (a.qk_norm) gk.load(a.k_norm, lrow);
            float gk_lo[RP::NP], gk_hi[RP::NP];
            gk.get(a.qk_norm, gk_lo, gk_hi);
            const int r = 4 * wid + lgrp;
            for (int i = 0; i < n_items; ++i) {
                const int j = 16 * i + r;
                const bool live = j < W && j < nrows;
                const int jj = live ? j : 0;                       // dead rows read a valid row
                const float* ks = qkv_b + (size_t)jj * row_stride + (size_t)a.n_q * HD + (size_t)g * HD;
                const float* vs = ks + (size_t)a.n_kv * HD;
                RP rk;
                rk.load(ks, a.rope + (size_t)(t + jj) * HALF, lrow);
                const typename RP::fv vlo = *(const typename RP::fv*)(vs + RP::NP * lrow);
                const typename RP::fv vhi = *(const typename RP::fv*)(vs + HALF + RP::NP * lrow);
                T klo[RP::NP], khi[RP::NP];
                rk.values(live, gk_lo, gk_hi, a.qk_norm, a.eps, klo, khi);
                T vl[RP::NP], vh[RP::NP];
#pragma unroll
                for (int p = 0; p < RP::NP; ++p) {
                    vl[p] = from_f32<T>(live ? vlo[p] : 0.f);
                    vh[p] = from_f32<T>(live ? vhi[p] : 0.f);
                }
                // the lane's dims 4 lrow .. 4 lrow + 3 (and + HALF) of key row r:
                // one 8-byte run of the K block (kblock_elem), four V elements
                // 4 apart (vblock_elem); the high half 1024 elements on
                const int ko = ((lrow / 8) * 64 + ((lrow % 8) / 2) * 16 + r) * 8 + 4 * (lrow % 2);
                const int vo = ((lrow / 4) * 64 + (r / 4) * 16 + 4 * (lrow % 4)) * 4 + r % 4;
                auto put = [&](T* kb, T* vb, int ko_, int vo_) {
                    uint2 k2, h2;
                    __builtin_memcpy(&k2, klo, 8);
                    __builtin_memcpy(&h2, khi, 8);
                    *(uint2*)(kb + ko_) = k2;
                    *(uint2*)(kb + ko_ + 1024) = h2;
#pragma unroll
                    for (int p = 0; p < RP::NP; ++p) {
                        vb[vo_ + 4 * p] = vl[p];
                        vb[vo_ + 4 * p + 1024] = vh[p];
                    }
                };
                put((T*)(smem + (size_t)i * BLK), (T*)(smem + (size_t)i * BLK + BLK / 2), ko, vo);
                if (live && j < a.kv_rows) {
                    const int pos = t + j, kr = pos % 16;
                    put((T*)a.kcache + head + (size_t)(pos / 16) * 16 * HD, (T*)a.vcache + head + (size_t)(pos / 16) * 16 * HD,
                        ko + (kr - r) * 8, vo + (kr / 4 - r / 4) * 64 + (kr % 4 - r % 4));
                }
            }
        }
        lds_sync();
    }

    f32x4 o_acc[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o_acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -1e30f, l_run = 0.f;
    const int jq = q % W;                                      // block row of this query column
    for (int it = 0; it < n_items; ++it) {
        const unsigned char* cur = blk ? smem + (size_t)it * BLK : kv_l + (size_t)(it & 1) * BLK;
        // scores of the block's 16 keys for this wave's query column lrow
        // (lane: keys 4 lgrp .. 4 lgrp + 3), scaled through the query rows
        f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds) mma_frag<T>(sc, *(const uint4*)(cur + ds * 1024 + lane * 16), qf[ds]);
        // The maximum below reads the scores right after the branch around the
        // key mask.  The compiler's wait states before that read do not cover
        // the branch-taken path (the read came two instructions after the last
        // MFMA), and the rescale vote then saw unfinished scores now and then:
        // results that changed from run to run.  Explicit wait states here.
        mfma_settle();
        float sv[4] = {sc[0], sc[1], sc[2], sc[3]};
        if (blk) {
            // block key kk is seen by block row jq iff kk <= jq or jq >= full_from
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int kk = it * 16 + lgrp * 4 + e;
                if (!((kk < nrows) & ((kk <= jq) | (jq >= a.full_from)))) sv[e] = -INFINITY;
            }
        } else {
            const int key0 = (kb_first + it) * 16;
            if (key0 + 16 > k_hi) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (key0 + lgrp * 4 + e >= k_hi) sv[e] = -INFINITY;
            }
        }
        // lazy reference maximum (k_attn's rule): raised, with the output and
        // sum rescaled, only when a score exceeds it by RESCALE_SLACK
        bool over = it == 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) over = over | (sv[e] > m_run + RESCALE_SLACK);
        if (__any(over)) {
            const float mloc = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
            const float m_new = fmaxf(m_run, xrow_max(mloc));
            const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
            l_run *= corr;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) o_acc[dt] *= corr;
            m_run = m_new;
        }
        f32x4 pw;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            pw[e] = __builtin_amdgcn_exp2f(sv[e] - m_run);
            l_run += pw[e];
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
            mma_k4(o_acc[dt], *(const vraw*)(cur + BLK / 2 + (dt * WAVE + lane) * sizeof(vraw)), pw);
        // explicit wait states after the P.V chain: the staging code below may
        // take the chain's accumulator source registers as temporaries
        mfma_settle();
        // prefix splits: the next block into the other buffer (read by every
        // wave in the previous turn, released by its barrier), the one after
        // into registers
        if (stager && !blk && it + 1 < n_items) {
            swrite((it + 1) & 1);
            if (it + 2 < n_items) gload(it + 2);
        }
        lds_sync();
    }
    l_run = xrow_sum(l_run);

    // partial of this split for the wave's query rows: max (log2 domain), sum,
    // unnormalised output
    if (q < QR) {
        const int gi = q / W, j = q % W;
        const size_t pr = (((size_t)b * a.n_q + g * G + gi) * W + j) * a.s_launch + s;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) *(f32x4*)(a.part_o + pr * HD + dt * 16 + lgrp * 4) = o_acc[dt];
        if (lgrp == 0) {
            a.part_ml[pr * 2 + 0] = m_run;
            a.part_ml[pr * 2 + 1] = l_run;
        }
    }
}

bool attn_rows_fits(int dtype, int head_dim, int qt, int chunk, int W) {
    return dtype == PBD_DTYPE_BF16 && head_dim == 128 && (qt == 4 || qt == 5) && !chunk && W <= ATTN_ROWS_WMAX;
}

hipError_t launch_attn_rows(const AttnArgs& a, int qt, int batch, hipStream_t st) {
    if (a.n_qgrp != 1 || a.chunk || a.W > ATTN_ROWS_WMAX || a.G * a.W > qt * 16) return hipErrorInvalidValue;
    const size_t smem = ((size_t)qt * 16 * (128 + 8) * 2 + 15) / 16 * 16 + 2 * 8192;
    const dim3 grid(a.s_launch, a.n_kv, batch);
    if (qt == 4) PBD_LAUNCH(k_attn_rows<4>, grid, dim3(4 * 64), smem, st, a);
    else if (qt == 5) PBD_LAUNCH(k_attn_rows<5>, grid, dim3(5 * 64), smem, st, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Tied LM head with the final RMSNorm folded in and a fused argmax.
//
// Each work-group keeps its waves' slices of the operand (all block rows) in
// registers and walks vocabulary tiles with a grid stride; the next tile's
// weight fragments are in flight while the current tile is reduced, so the
// 16-row tiles of the embedding matrix stream back to back.  Each work-group
// leaves one (max, argmax) per row; ties go to the lowest token id.  With
// CONF it also leaves the row's softmax partial over its tiles (maximum and
// sum of exp(value - maximum)), kept online by all 256 threads, two columns
// of each tile per thread.
// ---------------------------------------------------------------------------
constexpr int LM_FPW = 8;      // weight fragments per wave and tile (hidden <= 4 * 8 * FK)

template <typename T, bool SPLIT, bool CONF>
__global__ __launch_bounds__(256, 2) void k_lmhead(FGemmArgs a) {
    constexpr int NW = 4, MGH = 2;
    __shared__ f32x4 s_red[NW][MGH][WAVE];
    __shared__ float s_tile[MGH][16][17];
    __shared__ float s_rm[MGH * 16];
    __shared__ float s_sq[256];
    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    const int lrow = lane % 16;
    const int kb = a.kb;
    // r_m of every row from the sum-of-squares partials
    {
        const int row = threadIdx.x % 32, slice = threadIdx.x / 32;
        float sp = 0.f;
        if (row < a.M)
            for (int p = slice; p < a.n_sq; p += 8) sp += a.sq[(size_t)p * a.sq_stride + row];
        s_sq[threadIdx.x] = sp;
    }
    // operand slices in registers
    uint4 xh[LM_FPW][MGH], xl[LM_FPW][MGH];
#pragma unroll
    for (int i = 0; i < LM_FPW; ++i) {
        const int f = wid + NW * i;
#pragma unroll
        for (int mt = 0; mt < MGH; ++mt) {
            xh[i][mt] = uint4{0, 0, 0, 0};
            xl[i][mt] = uint4{0, 0, 0, 0};
            if (f < kb && mt < a.MT && mt * 16 + lrow < a.M) {
                const size_t xi = ((size_t)f * a.MT + mt) * WAVE + lane;
                xh[i][mt] = a.xhi[xi];
                if (SPLIT) xl[i][mt] = a.xlo[xi];
            }
        }
    }
    __syncthreads();
    if (threadIdx.x < 32) {
        float t = 0.f;
        for (int sl = 0; sl < 8; ++sl) t += s_sq[sl * 32 + threadIdx.x];
        s_rm[threadIdx.x] = a.n_sq > 0 ? rsqrtf(t / (float)a.norm_dim + a.eps) : 1.f;
    }
    float best = -INFINITY;
    int bi = 0x7fffffff;
    // the token id this thread's row excludes from its argmax (-1: none)
    const int excl = (int)threadIdx.x % a.W >= a.excl_from ? a.exclude : -1;
    float cmx = -INFINITY, csum = 0.f;     // CONF: running softmax partial of (row, column pair)
    const int crow = threadIdx.x % 32, ccol = (threadIdx.x / 32) * 2;
    uint4 wv[LM_FPW], wn[LM_FPW];
    auto load_tile = [&](int tile, uint4* dst) {
        const uint4* wt = a.w + (size_t)tile * kb * WAVE;
#pragma unroll
        for (int i = 0; i < LM_FPW; ++i) {
            const int f = wid + NW * i;
            dst[i] = (f < kb) ? wt[(size_t)f * WAVE + lane] : uint4{0, 0, 0, 0};
        }
    };
    int tile = blockIdx.x;
    if (tile < a.n_tiles) load_tile(tile, wv);
    for (; tile < a.n_tiles; tile += gridDim.x) {
        const int next = tile + gridDim.x;
        if (next < a.n_tiles) load_tile(next, wn);
        f32x4 acc[MGH];
#pragma unroll
        for (int mt = 0; mt < MGH; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < LM_FPW; ++i)
#pragma unroll
            for (int mt = 0; mt < MGH; ++mt) {
                mma_frag<T>(acc[mt], wv[i], xh[i][mt]);
                if (SPLIT) mma_frag<T>(acc[mt], wv[i], xl[i][mt]);
            }
#pragma unroll
        for (int mt = 0; mt < MGH; ++mt) s_red[wid][mt][lane] = acc[mt];
        __syncthreads();
        for (int idx = threadIdx.x; idx < MGH * WAVE * 4; idx += blockDim.x) {
            const int mt = idx / (WAVE * 4), ln = (idx / 4) % WAVE, e = idx % 4;
            const float v = s_red[0][mt][ln][e] + s_red[1][mt][ln][e] + s_red[2][mt][ln][e] + s_red[3][mt][ln][e];
            s_tile[mt][(ln / 16) * 4 + e][ln % 16] = v * s_rm[mt * 16 + ln % 16];
        }
        __syncthreads();
        if (threadIdx.x < MGH * 16) {
            const int m = threadIdx.x, mt = m / 16, ml = m % 16;
            if (m < a.M) {
                for (int n = 0; n < 16; ++n) {
                    const int v = tile * 16 + n;
                    const float val = s_tile[mt][n][ml];
                    if (a.logits) a.logits[(size_t)m * a.ldo + v] = val;
                    if (v == excl) continue;
                    if (val > best) { best = val; bi = v; }   // tiles ascend within a work-group
                }
            }
        }
        if (CONF && crow < a.M) {
            const float v0 = s_tile[crow / 16][ccol][crow % 16];
            const float v1 = s_tile[crow / 16][ccol + 1][crow % 16];
            const float nm = fmaxf(cmx, fmaxf(v0, v1));
            if (nm > -INFINITY) {
                csum = csum * expf(cmx - nm) + expf(v0 - nm) + expf(v1 - nm);
                cmx = nm;
            }
        }
#pragma unroll
        for (int i = 0; i < LM_FPW; ++i) wv[i] = wn[i];
    }
    if (threadIdx.x < a.M && threadIdx.x < MGH * 16) {
        a.arg_val[(size_t)blockIdx.x * a.M + threadIdx.x] = best;
        a.arg_idx[(size_t)blockIdx.x * a.M + threadIdx.x] = bi;
    }
    if (CONF) {
        // merge the eight column-pair partials of each row
        __syncthreads();
        float* s_mx = s_sq;
        float* s_sm = &s_tile[0][0][0];
        static_assert(MGH * 16 * 17 >= 256, "LDS reuse");
        s_mx[threadIdx.x] = cmx;
        s_sm[threadIdx.x] = csum;
        __syncthreads();
        if (threadIdx.x < 32 && (int)threadIdx.x < a.M) {
            float mx = -INFINITY;
            for (int k = 0; k < 8; ++k) mx = fmaxf(mx, s_mx[k * 32 + threadIdx.x]);
            float sm = 0.f;
            if (mx > -INFINITY)
                for (int k = 0; k < 8; ++k) {
                    const float pm = s_mx[k * 32 + threadIdx.x];
                    if (pm > -INFINITY) sm += s_sm[k * 32 + threadIdx.x] * expf(pm - mx);
                }
            a.arg_mx[(size_t)blockIdx.x * a.M + threadIdx.x] = mx;
            a.arg_sum[(size_t)blockIdx.x * a.M + threadIdx.x] = sm;
        }
    }
}

// Merge the split-KV partials of one (block row, query head) and write the
// O-projection operand.  Every one of the s_launch splits is read (unused ones
// carry max -inf and contribute nothing), so no load waits for the sequence's
// position; SMAX > 0: all loads issued at once.  A work-group takes
// blockDim.y block rows of one head (head_dim / EPL threads per row), so that
// its waves are full.
template <typename T, int SMAX>
__global__ __launch_bounds__(256) void k_combine(CombineArgs a) {
    // thread: EPL consecutive dims d0.. of head h for block row m
    constexpr int EPL = Elt<T>::EPL;
    const int m = blockIdx.x * blockDim.y + threadIdx.y, h = blockIdx.y, d0 = threadIdx.x * EPL;
    if (m >= a.M) return;
    const int b = m / a.W, j = m % a.W;
    const size_t pr0 = (((size_t)b * a.n_q + h) * a.W + j) * a.s_launch;
    float L = 0.f, o[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) o[i] = 0.f;
    auto add = [&](float wgt, const float4* src) {
#pragma unroll
        for (int q = 0; q < EPL / 4; ++q) {
            const float4 v = src[q];
            o[4 * q] += wgt * v.x;
            o[4 * q + 1] += wgt * v.y;
            o[4 * q + 2] += wgt * v.z;
            o[4 * q + 3] += wgt * v.w;
        }
    };
    if (SMAX > 0) {
        float ms[SMAX > 0 ? SMAX : 1], ls[SMAX > 0 ? SMAX : 1];
        float4 ov[SMAX > 0 ? SMAX : 1][EPL / 4];
#pragma unroll
        for (int s = 0; s < SMAX; ++s) {
            const int sc = s < a.s_launch ? s : 0;        // valid index; weight 0 below
            ms[s] = a.part_ml[(pr0 + sc) * 2];
            ls[s] = a.part_ml[(pr0 + sc) * 2 + 1];
#pragma unroll
            for (int q = 0; q < EPL / 4; ++q) ov[s][q] = ((const float4*)(a.part_o + (pr0 + sc) * a.head_dim + d0))[q];
        }
        float mx = -1e30f;
#pragma unroll
        for (int s = 0; s < SMAX; ++s)
            if (s < a.s_launch) mx = fmaxf(mx, ms[s]);
#pragma unroll
        for (int s = 0; s < SMAX; ++s) {
            if (s >= a.s_launch || !(ms[s] > -INFINITY)) continue;
            const float wgt = exp2f(ms[s] - mx);
            L += wgt * ls[s];
            add(wgt, ov[s]);
        }
    } else {
        // many splits: groups of eight loaded at once, merged online (the
        // running maximum raised between groups, the sums rescaled)
        float mx = -INFINITY;
        for (int s0 = 0; s0 < a.s_launch; s0 += 8) {
            float ms[8], ls[8];
            float4 ov[8][EPL / 4];
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int sc = min(s0 + c, a.s_launch - 1);     // valid index; masked below
                ms[c] = s0 + c < a.s_launch ? a.part_ml[(pr0 + sc) * 2] : -INFINITY;
                ls[c] = a.part_ml[(pr0 + sc) * 2 + 1];
#pragma unroll
                for (int q = 0; q < EPL / 4; ++q) ov[c][q] = ((const float4*)(a.part_o + (pr0 + sc) * a.head_dim + d0))[q];
            }
            float mg = mx;
#pragma unroll
            for (int c = 0; c < 8; ++c) mg = fmaxf(mg, ms[c]);
            if (!(mg > -INFINITY)) continue;
            if (mx > -INFINITY && mg > mx) {
                const float f = exp2f(mx - mg);
                L *= f;
#pragma unroll
                for (int i = 0; i < EPL; ++i) o[i] *= f;
            }
            mx = mg;
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                if (!(ms[c] > -INFINITY)) continue;
                const float wgt = exp2f(ms[c] - mx);
                L += wgt * ls[c];
                add(wgt, ov[c]);
            }
        }
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
    for (int i = 0; i < EPL; ++i) o[i] *= inv;
    put_operand_run<T>((T*)a.op_hi, (T*)a.op_lo, xfrag_elem<T>(m, h * a.head_dim + d0, a.MT), o, a.op_f16 != 0);
}

// ---------------------------------------------------------------------------
// Final argmax over the LM-head tile partials (ties: lowest id) and routing of
// the result: draft tokens (rows 1..D), verify tokens (rows 0..D), or the
// prefill's first generated token.
// ---------------------------------------------------------------------------
// R rows per work-group and 256 / R tile groups: the partials are [tile][row],
// so with R = 8 (passes of many rows) a wave's load covers 8 consecutive rows
// of eight tiles (32-byte runs); with R = 1 (few rows) all 256 threads share
// one row's tiles.  Each tile group keeps a running best over its tiles in
// order; a fixed tree over the groups merges them.
template <int R>
__global__ __launch_bounds__(256) void k_argmax(ArgmaxArgs a) {
    constexpr int TG = 256 / R;                 // tile groups
    const int r = threadIdx.x % R, tg = threadIdx.x / R;
    const int m = blockIdx.x * R + r;
    const bool live = m < a.M;
    const bool conf = a.conf != nullptr;
    float best = -INFINITY;
    int bi = 0x7fffffff;
    float mx = -INFINITY, sm = 0.f;      // softmax partial of the whole row (conf only)
    auto merge = [](float& m1, float& s1, float m2, float s2) {
        const float nm = fmaxf(m1, m2);
        if (nm == -INFINITY) return;
        s1 = (m1 > -INFINITY ? s1 * expf(m1 - nm) : 0.f) + (m2 > -INFINITY ? s2 * expf(m2 - nm) : 0.f);
        m1 = nm;
    };
    if (live) {
        // a group's tiles in order, eight tiles' loads issued together (the
        // index is clamped into range; tiles past the end are not merged)
        constexpr int U = 8;
        for (int t0 = tg; t0 < a.n_tiles; t0 += U * TG) {
            float v[U], cm[U], cs[U];
            int ix[U];
            size_t e[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                e[u] = (size_t)min(t0 + u * TG, a.n_tiles - 1) * a.M + m;
                v[u] = a.arg_val[e[u]];
                ix[u] = a.arg_idx[e[u]];
            }
            if (conf) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    cm[u] = a.arg_mx[e[u]];
                    cs[u] = a.arg_sum[e[u]];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (t0 + u * TG >= a.n_tiles) break;
                if (v[u] > best || (v[u] == best && ix[u] < bi)) { best = v[u]; bi = ix[u]; }
                if (conf) merge(mx, sm, cm[u], cs[u]);
            }
        }
    }
    __shared__ float s_v[TG][R];
    __shared__ int s_i[TG][R];
    __shared__ float s_m[TG][R], s_s[TG][R];
    s_v[tg][r] = best;
    s_i[tg][r] = bi;
    s_m[tg][r] = mx;
    s_s[tg][r] = sm;
    __syncthreads();
    for (int st = TG / 2; st > 0; st >>= 1) {
        if (tg < st) {
            const float v2 = s_v[tg + st][r];
            const int i2 = s_i[tg + st][r];
            if (v2 > s_v[tg][r] || (v2 == s_v[tg][r] && i2 < s_i[tg][r])) {
                s_v[tg][r] = v2;
                s_i[tg][r] = i2;
            }
            if (conf) {
                float m1 = s_m[tg][r], s1 = s_s[tg][r];
                merge(m1, s1, s_m[tg + st][r], s_s[tg + st][r]);
                s_m[tg][r] = m1;
                s_s[tg][r] = s1;
            }
        }
        __syncthreads();
    }
    if (tg != 0 || !live) return;
    best = s_v[0][r];
    bi = s_i[0][r];
    mx = s_m[0][r];
    sm = s_s[0][r];
    const int b = m / a.W, j = m % a.W;
    const int tok = bi;
    // a sequence the pass skipped (capacity: no rows assembled) keeps its
    // outputs untouched, as its cache rows are
    if (a.mode != PASS_PREFILL && a.nrows[b] == 0) return;
    if (a.mode == PASS_DRAFT) {
        const int nd = a.W - a.lead;
        if (j >= a.lead) {
            a.out[b * nd + j - a.lead] = tok;
            // log-probability of the argmax under the softmax of the whole row
            if (conf) a.conf[b * nd + j - a.lead] = best - (mx + logf(sm));
        } else if (a.out0) {
            a.out0[(size_t)b * a.out0_stride] = tok;
        }
    } else if (a.mode == PASS_VERIFY) {
        a.out[b * a.out_stride + a.out_off + j] = tok;
    } else if (a.compact) {
        const int r = a.lengths[m] - 1 - a.chunk_pos;  // row m: sequence m's gathered last row
        if (r >= 0 && r < a.nrows[m]) {
            a.out[m] = tok;                     // anchor
            a.seq_len_out[m] = a.lengths[m];
        }
    } else {
        if (a.chunk_pos + j == a.lengths[b] - 1 && j < a.nrows[b]) {
            a.out[b] = tok;                     // anchor
            a.seq_len_out[b] = a.lengths[b];
        }
    }
}

// One remasking pass of multi-step denoising (the denoising-steps ablation of
// Sec. 4.4 / Sec. 5.3; the remasking rule is a reading: the paper gives none).
// One wave per sequence, one lane per block position: a still-masked position
// is fixed when fewer than n_fix other still-masked positions beat it (higher
// confidence, or equal confidence and a lower position).  All lanes read the
// block state before any lane writes it.
__global__ __launch_bounds__(64) void k_remask(RemaskArgs a) {
    __shared__ float s_c[64];
    __shared__ int s_open[64];
    const int b = blockIdx.x, j = threadIdx.x;
    const size_t idx = (size_t)b * a.D + j;
    const bool open = j < a.D && a.block[idx] == a.mask_id;
    float c = open ? a.cand_conf[idx] : -INFINITY;
    if (c != c) c = -INFINITY;            // a NaN confidence ranks last
    s_c[j] = c;
    s_open[j] = open ? 1 : 0;
    __syncthreads();
    if (!open) return;
    int rank = 0;
    for (int i = 0; i < a.D; ++i)
        if (s_open[i] && (s_c[i] > c || (s_c[i] == c && i < j))) ++rank;
    if (rank < a.n_fix) {
        a.block[idx] = a.cand[idx];
        if (a.conf) a.conf[idx] = a.cand_conf[idx];
        if (a.fixed_at) a.fixed_at[idx] = a.step;
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
    // the passes' own bound (t + D + 1 <= max_seq): a sequence whose verify was
    // skipped for capacity commits nothing from its unwritten rows
    if (t < 0 || t + W > a.max_seq) { atomicOr(a.status, PBD_STATUS_CAPACITY); return; }
    for (int i = 0; i < W; ++i)
        a.out[b * W + i] = i < n ? a.draft[b * D + i] : (i == n ? a.verify[b * W + n] : -1);
    a.n_acc[b] = n;
    a.seq_len[b] = t + n + 1;
    a.anchor[b] = a.verify[b * W + n];
}

// ---------------------------------------------------------------------------
// Initialisation helpers
// ---------------------------------------------------------------------------
// Row of source matrix for row `row` of packed tile `tile`.
static __device__ __forceinline__ void map_row(int row_map, int n_src, const int* src_rows, int tile, int row,
                                               int& src, int& srow) {
    if (row_map == MAP_INTERLEAVE2) {
        src = row < 8 ? 0 : 1;
        srow = tile * 8 + (row % 8);
    } else {
        const int r = tile * 16 + row;
        src = 0;
        srow = r;
        if (n_src > 1 && r >= src_rows[0]) { src = 1; srow = r - src_rows[0]; }
        if (n_src > 2 && r >= src_rows[0] + src_rows[1]) { src = 2; srow = r - src_rows[0] - src_rows[1]; }
    }
}

// Repack [rows][K] matrices into 16-row fragment tiles.
template <typename T>
__global__ void k_pack(PackArgs a) {
    constexpr int EPL = Elt<T>::EPL;
    constexpr int FK = Elt<T>::FK;
    const size_t total = (size_t)a.n_tiles * a.kb * WAVE;
    for (size_t id = blockIdx.x * (size_t)blockDim.x + threadIdx.x; id < total; id += (size_t)gridDim.x * blockDim.x) {
        const int lane = id % WAVE;
        const int f = (id / WAVE) % a.kb;
        const int tile = id / ((size_t)WAVE * a.kb);
        const int row = lane % 16, grp = lane / 16;
        int src, srow;
        map_row(a.row_map, a.n_src, a.src_rows, tile, row, src, srow);
        T* dst = (T*)a.dst + id * EPL;
        const bool live = tile * 16 + row < a.rows_total && srow < a.src_rows[src];
        const T* Wsrc = (const T*)a.w[src] + (size_t)srow * a.K + f * FK + grp * EPL;
#pragma unroll
        for (int e = 0; e < EPL; ++e) dst[e] = live ? Wsrc[e] : from_f32<T>(0.f);
    }
}

// Repack LoRA B [rows][r] into expand blocks: block (tile, t), lane (row n, group g)
// holds B[row(n)][16 t + 4 g .. +4].
template <typename T>
__global__ void k_pack_expand(PackExpandArgs a) {
    const size_t total = (size_t)a.n_tiles * a.rt * WAVE;
    for (size_t id = blockIdx.x * (size_t)blockDim.x + threadIdx.x; id < total; id += (size_t)gridDim.x * blockDim.x) {
        const int lane = id % WAVE;
        const int t = (id / WAVE) % a.rt;
        const int tile = id / ((size_t)WAVE * a.rt);
        int src, srow;
        map_row(a.row_map, a.n_src, a.src_rows, tile, lane % 16, src, srow);
        const int k0 = 16 * t + 4 * (lane / 16);
        T* dst = (T*)a.dst + id * 4;
        for (int e = 0; e < 4; ++e)
            dst[e] = (k0 + e < a.r && srow < a.src_rows[src]) ? ((const T*)a.b[src])[(size_t)srow * a.r + k0 + e]
                                                             : from_f32<T>(0.f);
    }
}

__global__ void k_fill_u32(uint32_t* p, size_t n, uint32_t v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// fp16 copy of packed bf16 data (two values per word, round to nearest even;
// exact for magnitudes in [2^-14, 65504])
__global__ void k_bf16_to_f16(const uint32_t* src, uint32_t* dst, size_t n) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        const uint32_t u = src[i];
        const _Float16 lo = (_Float16)__uint_as_float(u << 16), hi = (_Float16)__uint_as_float(u & 0xffff0000u);
        dst[i] = (uint32_t)__builtin_bit_cast(unsigned short, lo) | ((uint32_t)__builtin_bit_cast(unsigned short, hi) << 16);
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------
// one (epilogue, m-group, rank tiles) instance; instances whose m-group
// exceeds the shrink-accumulator cap are never launched (fgemm_mgroup) and
// not instantiated
template <typename T, bool SPLIT, int EPI, int MG, int LRT>
static hipError_t launch_fgemm_inst(const FGemmArgs& a, hipStream_t st) {
    if constexpr (MG <= FG<EPI>::mg_cap(LRT)) {
        PBD_LAUNCH((k_fgemm<T, EPI, MG, SPLIT, LRT>), dim3(a.n_tiles * a.ksplit), dim3(FG<EPI>::NW * 64), 0, st, a);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

template <typename T, bool SPLIT, int EPI, int MG>
static hipError_t launch_fgemm_lrt(const FGemmArgs& a, int lrt, hipStream_t st) {
    switch (lrt) {
        case 0: return launch_fgemm_inst<T, SPLIT, EPI, MG, 0>(a, st);
        case 1: return launch_fgemm_inst<T, SPLIT, EPI, MG, 1>(a, st);
        case 2: return launch_fgemm_inst<T, SPLIT, EPI, MG, 2>(a, st);
        case 3: return launch_fgemm_inst<T, SPLIT, EPI, MG, 3>(a, st);
        case 4: return launch_fgemm_inst<T, SPLIT, EPI, MG, 4>(a, st);
        default: return hipErrorInvalidValue;
    }
}

template <typename T, bool SPLIT>
static hipError_t launch_fgemm_t(const FGemmArgs& a, int epi, int mg, hipStream_t st) {
    const int lrt = (a.lora && epi != EPI_ARGMAX) ? a.rt : 0;
#define PBD_FG_CASE(E, G) \
    if (epi == E && mg == G) return launch_fgemm_lrt<T, SPLIT, E, G>(a, lrt, st);
    PBD_FG_CASE(EPI_STORE, 1) PBD_FG_CASE(EPI_STORE, 2) PBD_FG_CASE(EPI_STORE, 4)
    PBD_FG_CASE(EPI_RESID, 1) PBD_FG_CASE(EPI_RESID, 2)
    PBD_FG_CASE(EPI_SWIGLU, 1) PBD_FG_CASE(EPI_SWIGLU, 2) PBD_FG_CASE(EPI_SWIGLU, 4)
#undef PBD_FG_CASE
    if (epi == EPI_ARGMAX) {
        const dim3 grid(a.n_tiles * a.ksplit), block(FG<EPI_ARGMAX>::NW * 64);
        switch (mg) {
            case 1: PBD_LAUNCH((k_fgemm<T, EPI_ARGMAX, 1, SPLIT, 0>), grid, block, 0, st, a); break;
            case 2: PBD_LAUNCH((k_fgemm<T, EPI_ARGMAX, 2, SPLIT, 0>), grid, block, 0, st, a); break;
            case 4: PBD_LAUNCH((k_fgemm<T, EPI_ARGMAX, 4, SPLIT, 0>), grid, block, 0, st, a); break;
            case 8: PBD_LAUNCH((k_fgemm<T, EPI_ARGMAX, 8, SPLIT, 0>), grid, block, 0, st, a); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    return hipErrorInvalidValue;
}

int fgemm_threads(int epi) {
    return epi == EPI_STORE ? FG<EPI_STORE>::NW * 64
         : epi == EPI_RESID ? FG<EPI_RESID>::NW * 64
         : epi == EPI_SWIGLU ? FG<EPI_SWIGLU>::NW * 64 : FG<EPI_ARGMAX>::NW * 64;
}

// m-tiles per pass over the weights: enough for the rows, bounded by the
// register budget (residual GEMMs hold the x slice; LoRA shrink partials
// grow with the rank tiles) and by LDS
int fgemm_mgroup(int epi, int MT, int lrt) {
    int cap = epi == EPI_ARGMAX ? 8 : (epi == EPI_RESID ? 2 : 4);
    const int lcap = epi == EPI_STORE ? FG<EPI_STORE>::mg_cap(lrt)
                   : epi == EPI_RESID ? FG<EPI_RESID>::mg_cap(lrt)
                   : epi == EPI_SWIGLU ? FG<EPI_SWIGLU>::mg_cap(lrt) : 8;
    cap = std::min(cap, lcap);
    int mg = 1;
    while (mg < MT && mg < cap) mg *= 2;
    return mg;
}

hipError_t launch_fgemm(int dtype, const FGemmArgs& a, int epi, hipStream_t st) {
    const int lrt = (a.lora && epi != EPI_ARGMAX) ? a.rt : 0;
    if (a.ksplit < 1 || a.ksplit > KSPLIT_MAX ||
        (a.ksplit > 1 && (!a.part || !a.cnt || a.MT > fgemm_mgroup(epi, a.MT, lrt))))
        return hipErrorInvalidValue;
    const int mg = fgemm_mgroup(epi, a.MT, lrt);
    // bf16 models always carry the operand as value + residual
    if (dtype == PBD_DTYPE_BF16) return a.xlo ? launch_fgemm_t<bf16, true>(a, epi, mg, st) : hipErrorInvalidValue;
    return launch_fgemm_t<float, false>(a, epi, mg, st);
}

bool lmhead_fits(int kb, int MT) { return kb <= 4 * LM_FPW && MT <= 2; }

hipError_t launch_lmhead(int dtype, const FGemmArgs& a, int grid, hipStream_t st) {
    const bool conf = a.arg_sum != nullptr;
    if (conf && !a.arg_mx) return hipErrorInvalidValue;
    if (dtype == PBD_DTYPE_BF16) {
        if (!a.xlo) return hipErrorInvalidValue;
        if (conf) PBD_LAUNCH((k_lmhead<bf16, true, true>), dim3(grid), dim3(256), 0, st, a);
        else PBD_LAUNCH((k_lmhead<bf16, true, false>), dim3(grid), dim3(256), 0, st, a);
    } else {
        if (conf) PBD_LAUNCH((k_lmhead<float, false, true>), dim3(grid), dim3(256), 0, st, a);
        else PBD_LAUNCH((k_lmhead<float, false, false>), dim3(grid), dim3(256), 0, st, a);
    }
    return hipGetLastError();
}

size_t attn_smem_main(int dtype, int head_dim, int qt) {
    const size_t es = dtype == PBD_DTYPE_BF16 ? 2 : 4;
    const size_t ldq = head_dim + 16 / es;
    const size_t ops = (qt * 16 * ldq + 48 * ldq + 48 * (size_t)head_dim) * es;
    const size_t ob = (size_t)2 * qt * 16 * (head_dim + 4) * 4;
    const size_t m = ops > ob ? ops : ob;
    return (m + 15) / 16 * 16;
}

size_t attn_smem_bytes(int dtype, int head_dim, int qt) {
    return attn_smem_main(dtype, head_dim, qt) + (size_t)4 * qt * 16 * 2 * 4;
}

template <typename T, int HD>
static hipError_t launch_attn_hd(const AttnArgs& a, int qt, dim3 grid, size_t smem, hipStream_t st) {
    switch (qt) {
        case 1: PBD_LAUNCH((k_attn<T, HD, 1>), grid, dim3(256), smem, st, a); break;
        case 2: PBD_LAUNCH((k_attn<T, HD, 2>), grid, dim3(256), smem, st, a); break;
        case 3: PBD_LAUNCH((k_attn<T, HD, 3>), grid, dim3(256), smem, st, a); break;
        case 4: PBD_LAUNCH((k_attn<T, HD, 4>), grid, dim3(256), smem, st, a); break;
        case 5: PBD_LAUNCH((k_attn<T, HD, 5>), grid, dim3(256), smem, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attn(int dtype, int head_dim, int qt, const AttnArgs& a, int batch, hipStream_t st) {
    dim3 grid(a.s_launch + a.pf_x, a.n_kv, batch * a.n_qgrp);
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

#define PBD_DISPATCH(dtype, KERNEL, grid, block, st, args)                                        \
    do {                                                                                          \
        if ((dtype) == PBD_DTYPE_BF16) PBD_LAUNCH(KERNEL<bf16>, grid, block, 0, st, args); \
        else PBD_LAUNCH(KERNEL<float>, grid, block, 0, st, args);                         \
        return hipGetLastError();                                                                 \
    } while (0)

hipError_t launch_assemble(int dtype, const AssembleArgs& a, int batch, hipStream_t st) {
    PBD_DISPATCH(dtype, k_assemble, dim3(a.W, batch), dim3(256), st, a);
}
template <typename T>
static hipError_t launch_combine_t(const CombineArgs& a_in, int M, hipStream_t st) {
    CombineArgs a = a_in;
    a.M = M;
    const int tx = a.head_dim / Elt<T>::EPL, rows = std::max(1, 256 / tx);   // rows per work-group
    const dim3 grid((M + rows - 1) / rows, a.n_q), block(tx, rows);
    if (a.s_launch <= 4) PBD_LAUNCH((k_combine<T, 4>), grid, block, 0, st, a);
    else if (a.s_launch <= 8) PBD_LAUNCH((k_combine<T, 8>), grid, block, 0, st, a);
    else PBD_LAUNCH((k_combine<T, 0>), grid, block, 0, st, a);
    return hipGetLastError();
}
hipError_t launch_combine(int dtype, const CombineArgs& a, int M, hipStream_t st) {
    return dtype == PBD_DTYPE_BF16 ? launch_combine_t<bf16>(a, M, st) : launch_combine_t<float>(a, M, st);
}
hipError_t launch_pack(int dtype, const PackArgs& a, hipStream_t st) {
    PBD_DISPATCH(dtype, k_pack, dim3(1024), dim3(256), st, a);
}
hipError_t launch_pack_expand(int dtype, const PackExpandArgs& a, hipStream_t st) {
    PBD_DISPATCH(dtype, k_pack_expand, dim3(256), dim3(256), st, a);
}
hipError_t launch_argmax(const ArgmaxArgs& a, hipStream_t st) {
    // eight rows per work-group at 256 rows or more (the tied LM head of 32
    // sequences x 33 rows over a 151936-token vocabulary, 1056 rows x 1187
    // tiles: 49 us, against 87 at sixteen rows, 105 at four and 143 at one)
    if (a.M >= 256) PBD_LAUNCH(k_argmax<8>, dim3((a.M + 7) / 8), dim3(256), 0, st, a);
    else PBD_LAUNCH(k_argmax<1>, dim3(a.M), dim3(256), 0, st, a);
    return hipGetLastError();
}
hipError_t launch_remask(const RemaskArgs& a, int batch, hipStream_t st) {
    if (a.D < 1 || a.D > 64 || batch < 1) return hipErrorInvalidValue;
    PBD_LAUNCH(k_remask, dim3(batch), dim3(64), 0, st, a);
    return hipGetLastError();
}
hipError_t launch_kvwrite(int dtype, int head_dim, const KVWriteArgs& a, int batch, hipStream_t st) {
    const dim3 grid((a.W + 15) / 16, a.n_kv, batch), block(256);
    if (dtype == PBD_DTYPE_BF16) {
        if (head_dim == 128) PBD_LAUNCH((k_kvwrite<bf16, 128>), grid, block, 0, st, a);
        else if (head_dim == 64) PBD_LAUNCH((k_kvwrite<bf16, 64>), grid, block, 0, st, a);
        else return hipErrorInvalidValue;
    } else {
        if (head_dim == 128) PBD_LAUNCH((k_kvwrite<float, 128>), grid, block, 0, st, a);
        else if (head_dim == 64) PBD_LAUNCH((k_kvwrite<float, 64>), grid, block, 0, st, a);
        else return hipErrorInvalidValue;
    }
    return hipGetLastError();
}
template <typename T>
__global__ __launch_bounds__(256) void k_gather_last(GatherArgs a) {
    constexpr int EPL = Elt<T>::EPL, FK = Elt<T>::FK;
    const int b = blockIdx.x;
    const int r = a.lengths[b] - 1 - a.chunk_pos;
    const int row = (r >= 0 && r < a.nrows[b]) ? r : 0;  // out of this chunk: any valid row (unused)
    const int m = b * a.W + row;
    for (int idx = threadIdx.x; idx < a.kb * (FK / EPL); idx += blockDim.x) {
        const int f = idx / (FK / EPL), k = (idx % (FK / EPL)) * EPL;
        const size_t src = frag_elem<T>((size_t)f * a.MT + m / 16, m % 16, k);
        const size_t dst = frag_elem<T>((size_t)f * a.MTc + b / 16, b % 16, k);
        *(uint4*)((T*)a.c_hi + dst) = *(const uint4*)((const T*)a.x_hi + src);
        if (a.x_lo) *(uint4*)((T*)a.c_lo + dst) = *(const uint4*)((const T*)a.x_lo + src);
    }
    for (int p = threadIdx.x; p < a.n_sq; p += blockDim.x) a.c_sq[(size_t)p * a.sqc_stride + b] = a.sq[(size_t)p * a.sq_stride + m];
}

hipError_t launch_gather_last(int dtype, const GatherArgs& a, int batch, hipStream_t st) {
    if (dtype == PBD_DTYPE_BF16) PBD_LAUNCH(k_gather_last<bf16>, dim3(batch), dim3(256), 0, st, a);
    else PBD_LAUNCH(k_gather_last<float>, dim3(batch), dim3(256), 0, st, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Large-M projection (prefill chunks, passes of many block rows).  The skinny
// GEMM above streams each weight tile once against every row; with hundreds of
// rows it would re-read the operand per weight tile and wait a full load
// latency per 64-row group.
// Here a work-group owns a 64-row x 64-column output block (4 x 4 MFMA tiles,
// a 2 x 2 tile quadrant per wave) and walks K through a double buffer in LDS:
// each K step's 4 W and 4 (+4 residual) operand fragments are loaded once by
// the work-group, four steps ahead, and every wave reads its quadrant's
// fragments from LDS.  r_m (the folded RMSNorm) scales rows in the epilogue
// and the fp32 result goes to out.  Residual and SwiGLU epilogues run after
// it as row kernels.  Loads are unconditional from clamped addresses (a
// guarded load would make the compiler wait for every load at each loop
// turn): tiles past the ends only feed outputs that are not stored, steps
// past K are not computed.  With the adapter, a first launch of this kernel on the stacked
// LoRA A tiles leaves the shrink u = A x in fp32, and the projection adds
// s * B u per tile before the r_m scaling (r_m (W x + s B A x), the same sum
// the skinny GEMM forms in-tile).
// ---------------------------------------------------------------------------
// WT: tiles per wave in each direction (2: 64x64 blocks, 4: 128x128 blocks);
// H16: fp16 operands and fp16 weight fragments (bf16 models), one MFMA per
// fragment pair and fp16 operands written by the epilogues
template <typename T, bool SPLIT, int WT, bool H16>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WT == 2 && H16 ? 5 : 1, 8))) void k_gemm_big(BigGemmArgs a) {
    static_assert(!H16 || (!SPLIT && sizeof(T) == 2), "fp16 operands replace the bf16 pair");
    constexpr int BT = 2 * WT;                  // m- and n-tiles per block
    constexpr int FPW = BT / 4;                 // fragments of each kind a wave stages per step
    constexpr int NSL = 256 / (BT * 16);        // RMSNorm partial slices per row
    const int lane = threadIdx.x % WAVE, wid = threadIdx.x / WAVE;
    const int lrow = lane % 16, lgrp = lane / 16;
    const int bm = a.m_fast ? blockIdx.x : blockIdx.y, bn = a.m_fast ? blockIdx.y : blockIdx.x;
    const int mt0 = bm * BT + (wid / 2) * WT, nt0 = bn * BT + (wid % 2) * WT;
    __shared__ float s_part[NSL][BT * 16];
    __shared__ float s_rm[BT * 16];
    int ntc[WT];
#pragma unroll
    for (int i = 0; i < WT; ++i) ntc[i] = min(nt0 + i, a.n_tiles - 1);
    // wave w loads fragments w FPW .. w FPW + FPW - 1 of each kind (W tile,
    // value and residual m-tile) GS steps ahead and writes them to one of two
    // LDS step buffers; all waves read their operands from there, so each
    // fragment leaves the cache once per work-group (native vectors keep the
    // slots in registers)
    constexpr int GS = 4;
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    __shared__ u32x4 s_op[2][3 * BT][WAVE];     // [W tiles | value m-tiles | residual m-tiles]
    int ntw[FPW], mtw[FPW];
#pragma unroll
    for (int k = 0; k < FPW; ++k) {
        ntw[k] = min(bn * BT + wid * FPW + k, a.n_tiles - 1);
        mtw[k] = min(bm * BT + wid * FPW + k, a.MT - 1);
    }
    u32x4 gv[GS][3][FPW];                 // W, value, residual fragments of a step
    // this work-group's K fragments [kf0, kf0 + nkf) (split-K: slice blockIdx.z)
    const int kper = a.kper > 0 ? a.kper : a.kb;
    const int kf0 = (int)blockIdx.z * kper, nkf = min(a.kb, kf0 + kper) - kf0;
    auto gload = [&](int f, int st) {
        const int fc = kf0 + min(f, nkf - 1);
#pragma unroll
        for (int k = 0; k < FPW; ++k) {
            gv[st][0][k] = *(const u32x4*)(a.w + ((size_t)ntw[k] * a.kb + fc) * WAVE + lane);
            const size_t xi = ((size_t)fc * a.MT + mtw[k]) * WAVE + lane;
            gv[st][1][k] = *(const u32x4*)(a.xhi + xi);
            if (SPLIT) gv[st][2][k] = *(const u32x4*)(a.xlo + xi);
        }
    };
    auto swrite = [&](int st, int buf) {
#pragma unroll
        for (int k = 0; k < FPW; ++k) {
            s_op[buf][wid * FPW + k][lane] = gv[st][0][k];
            s_op[buf][BT + wid * FPW + k][lane] = gv[st][1][k];
            if (SPLIT) s_op[buf][2 * BT + wid * FPW + k][lane] = gv[st][2][k];
        }
    };
#pragma unroll
    for (int st = 0; st < GS; ++st) gload(st, st);
    // RMSNorm partials of the block's rows: NSL slices per row, summed in LDS
    {
        const int r = threadIdx.x % (BT * 16), sl = threadIdx.x / (BT * 16);
        const int m = bm * BT * 16 + r;
        float sm = 0.f;
        if (m < a.M)
            for (int p = sl; p < a.n_sq; p += NSL) sm += a.sq[(size_t)p * a.sq_stride + m];
        s_part[sl][r] = sm;
    }
    f32x4 acc[WT][WT];
#pragma unroll
    for (int j = 0; j < WT; ++j)
#pragma unroll
        for (int i = 0; i < WT; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    // step f sits in LDS buffer f & 1 (GS is even, so that is u & 1); each
    // turn writes step f + 1 into the other buffer, reloads the register slot
    // of step f (already in LDS) with step f + GS, and ends with a barrier.
    // Loads past K repeat the last step; their products are not formed.
    swrite(0, 0);
    lds_sync();
    for (int f0 = 0; f0 < nkf; f0 += GS) {
#pragma unroll
        for (int u = 0; u < GS; ++u) {
            const int buf = u & 1;
            uint4 w2[WT], h2[WT], l2[WT];
#pragma unroll
            for (int i = 0; i < WT; ++i) w2[i] = __builtin_bit_cast(uint4, s_op[buf][(wid % 2) * WT + i][lane]);
#pragma unroll
            for (int j = 0; j < WT; ++j) {
                h2[j] = __builtin_bit_cast(uint4, s_op[buf][BT + (wid / 2) * WT + j][lane]);
                if (SPLIT) l2[j] = __builtin_bit_cast(uint4, s_op[buf][2 * BT + (wid / 2) * WT + j][lane]);
            }
            swrite((u + 1) % GS, buf ^ 1);
            gload(f0 + u + GS, u);
            if (f0 + u < nkf) {
#pragma unroll
                for (int j = 0; j < WT; ++j)
#pragma unroll
                    for (int i = 0; i < WT; ++i) {
                        if (H16) {
                            acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                                __builtin_bit_cast(f16x8, w2[i]), __builtin_bit_cast(f16x8, h2[j]), acc[j][i], 0, 0, 0);
                        } else {
                            mma_frag<T>(acc[j][i], w2[i], h2[j]);
                            if (SPLIT) mma_frag<T>(acc[j][i], w2[i], l2[j]);
                        }
                    }
            }
            lds_sync();
        }
    }
    if (a.lrt > 0) {
        // LoRA expand: lane operand u[m = tile row lrow][r = 16 t + 4 lgrp + e],
        // the layout the shrink's epilogue stored it in
        typedef typename K4<T>::raw braw;
        float lsc[WT];
        int mc[WT];
#pragma unroll
        for (int j = 0; j < WT; ++j) {
            const int m = (mt0 + j) * 16 + lrow;
            mc[j] = min(m, a.M - 1);
            lsc[j] = (m < a.M && m % a.W >= a.adapter_from) ? a.scale : 0.f;
        }
        const int nsrc = a.lora_mode == LORA_ROW_HALF ? 2 : 1;
        constexpr int LRT4 = 4;                  // rank tiles staged through LDS (r <= 64)
        if (WT == 2 && sizeof(T) == 2 && a.lrt <= LRT4) {
            // Stage the block's u rows and B fragments through the K loop's
            // LDS buffers (free after its last barrier), one LoRA source at a
            // time: every thread issues its share of the loads at once, so the
            // expand waits for memory once per source instead of once per rank
            // tile.  us[m-tile][t][row][16 r], bs[n-tile][t][lane] (16-bit B).
            static_assert(sizeof(s_op) >= (size_t)BT * LRT4 * 16 * 16 * 4 + (size_t)BT * LRT4 * WAVE * 8,
                          "u and B of a source fit the step buffers");
            float* us = (float*)&s_op[0][0][0];
            uint2* bs = (uint2*)(us + BT * LRT4 * 16 * 16);
            const int nt_first = min(bn * BT, a.n_tiles - 1), nt_last = min(bn * BT + BT - 1, a.n_tiles - 1);
            auto src_of = [&](int nt) {
                return a.lora_mode == LORA_BY_TILE ? (nt < a.tile_split0 ? 0 : nt < a.tile_split1 ? 1 : 2) : 0;
            };
            const int src_lo = src_of(nt_first), src_hi = src_of(nt_last) + nsrc - 1;
            // B fragments of the block's n-tiles (2 x 16 bytes per thread)
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int c = k * 256 + (int)threadIdx.x;      // 16-byte chunk: [n-tile][t][32 chunks]
                const int ib = c / (LRT4 * 32), t = (c / 32) % LRT4, q = c % 32;
                if (t < a.lrt) {
                    const int nt = min(bn * BT + ib, a.n_tiles - 1);
                    ((uint4*)bs)[c] = *(const uint4*)((const T*)a.lb + ((size_t)nt * a.lrt + t) * WAVE * 4 + q * 8);
                }
            }
            for (int src = src_lo; src <= src_hi; ++src) {
                __syncthreads();                         // the K loop's (or the last source's) reads are done
                // u of the block's 64 rows for this source (4 x 16 bytes per thread)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int c = k * 256 + (int)threadIdx.x;  // [m-tile][t][row][4 chunks]
                    const int jb = c / (LRT4 * 64), t = (c / 64) % LRT4, row = (c / 4) % 16, q = c % 4;
                    if (t < a.lrt) {
                        const int m = min((bm * BT + jb) * 16 + row, a.M - 1);
                        ((float4*)us)[c] = *(const float4*)(a.u + (size_t)m * a.ldu + (src * a.lrt + t) * 16 + q * 4);
                    }
                }
                __syncthreads();
#pragma unroll
                for (int i = 0; i < WT; ++i) {
                    const int ib = (wid % 2) * WT + i, s0 = src_of(ntc[i]);
                    const int sc = src - s0;
                    if (sc < 0 || sc >= nsrc) continue;
                    // gate/up tiles: rows 0-7 take source 0 (gate), 8-15 source 1 (up)
                    const bool zero = nsrc == 2 && ((lrow < 8) != (sc == 0));
                    for (int t = 0; t < a.lrt; ++t) {
                        const uint2 b = zero ? uint2{0u, 0u} : bs[(ib * LRT4 + t) * WAVE + lane];
#pragma unroll
                        for (int j = 0; j < WT; ++j) {
                            const int jb = (wid / 2) * WT + j;
                            const float4 uv = ((const float4*)us)[((jb * LRT4 + t) * 16 + lrow) * 4 + lgrp];
                            mma_k4_split(acc[j][i], b, f32x4{uv.x, uv.y, uv.z, uv.w} * lsc[j]);
                        }
                    }
                }
            }
        } else
#pragma unroll
        for (int i = 0; i < WT; ++i) {
            const int nt = ntc[i];
            const int s0 = a.lora_mode == LORA_BY_TILE ? (nt < a.tile_split0 ? 0 : nt < a.tile_split1 ? 1 : 2) : 0;
            for (int t = 0; t < a.lrt; ++t) {
                braw b;
                __builtin_memcpy(&b, (const T*)a.lb + (((size_t)nt * a.lrt + t) * WAVE + lane) * 4, sizeof(braw));
                for (int sc = 0; sc < nsrc; ++sc) {
                    // gate/up tiles: rows 0-7 take source 0 (gate), 8-15 source 1 (up)
                    const braw bb = (nsrc == 2 && ((lrow < 8) != (sc == 0))) ? braw{} : b;
#pragma unroll
                    for (int j = 0; j < WT; ++j) {
                        const float4 uv = *(const float4*)(a.u + (size_t)mc[j] * a.ldu + ((s0 + sc) * a.lrt + t) * 16 + lgrp * 4);
                        mma_k4_split(acc[j][i], bb, f32x4{uv.x, uv.y, uv.z, uv.w} * lsc[j]);
                    }
                }
            }
        }
    }
    __syncthreads();
    if (threadIdx.x < BT * 16) {
        float sm = 0.f;
#pragma unroll
        for (int sl = 0; sl < NSL; ++sl) sm += s_part[sl][threadIdx.x];
        s_rm[threadIdx.x] = a.n_sq > 0 ? rsqrtf(sm / (float)a.norm_dim + a.eps) : 1.f;
    }
    __syncthreads();
    // lane: row lrow of the m-tile, columns 4 lgrp .. 4 lgrp + 3 of the n-tile
    if (a.arg_val) {
        // every lane takes part in the cross-lane steps; only live rows store
#pragma unroll
        for (int j = 0; j < WT; ++j)
#pragma unroll
            for (int i = 0; i < WT; ++i) {
                const int mt = mt0 + j, nt = nt0 + i, m = mt * 16 + lrow;
                const bool live = mt < a.MT && m < a.M && nt < a.n_tiles;
                const f32x4 v = acc[j][i] * s_rm[m - bm * BT * 16];
                const int col0 = nt * 16 + lgrp * 4;
                if (live && a.logits) *(float4*)(a.logits + (size_t)m * a.ldo + col0) = float4{v[0], v[1], v[2], v[3]};
                const int excl = m % a.W >= a.excl_from ? a.exclude : -1;
                float best = -INFINITY;
                int bi = 0x7fffffff;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (col0 + e != excl && v[e] > best) { best = v[e]; bi = col0 + e; }   // ascending: first max wins
#pragma unroll
                for (int off = 16; off <= 32; off *= 2) {       // the row's four lane groups
                    const float ob = __shfl_xor(best, off);
                    const int oi = __shfl_xor(bi, off);
                    if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
                }
                if (a.arg_mx) {      // softmax partial over all 16 columns
                    float mx = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
                    mx = fmaxf(mx, __shfl_xor(mx, 16));
                    mx = fmaxf(mx, __shfl_xor(mx, 32));
                    float sm = expf(v[0] - mx) + expf(v[1] - mx) + expf(v[2] - mx) + expf(v[3] - mx);
                    sm += __shfl_xor(sm, 16);
                    sm += __shfl_xor(sm, 32);
                    if (live && lgrp == 0) {
                        a.arg_mx[(size_t)nt * a.M + m] = mx;
                        a.arg_sum[(size_t)nt * a.M + m] = sm;
                    }
                }
                if (live && lgrp == 0) {
                    a.arg_val[(size_t)nt * a.M + m] = best;
                    a.arg_idx[(size_t)nt * a.M + m] = bi;
                }
            }
        return;
    }
    if (a.rx) {
        // residual: the lane's 4 columns of the row; the tile's sum of squares
        // over its four lane groups; runs of EPL operand values gathered from
        // the neighbouring lane group for bf16
        constexpr int EPL = Elt<T>::EPL;
#pragma unroll
        for (int j = 0; j < WT; ++j)
#pragma unroll
            for (int i = 0; i < WT; ++i) {
                const int mt = mt0 + j, nt = nt0 + i, m = mt * 16 + lrow;
                const bool live = mt < a.MT && m < a.M && nt < a.n_tiles;
                const f32x4 v = acc[j][i] * s_rm[m - bm * BT * 16];
                const int col0 = nt * 16 + lgrp * 4;
                float xv[4] = {0.f, 0.f, 0.f, 0.f}, gv4[4] = {0.f, 0.f, 0.f, 0.f};
                if (live) {
                    float4* xp = (float4*)(a.rx + (size_t)m * a.ldx + col0);
                    const float4 xo = *xp;
                    xv[0] = xo.x + v[0]; xv[1] = xo.y + v[1]; xv[2] = xo.z + v[2]; xv[3] = xo.w + v[3];
                    *xp = float4{xv[0], xv[1], xv[2], xv[3]};
                    const T* g = (const T*)a.rgain + col0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) gv4[e] = to_f32(g[e]);
                }
                float ss = xv[0] * xv[0] + xv[1] * xv[1] + xv[2] * xv[2] + xv[3] * xv[3];
                ss += __shfl_xor(ss, 16);
                ss += __shfl_xor(ss, 32);
                float ov[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) ov[e] = xv[e] * gv4[e];
#pragma unroll
                for (int e = 0; e < 4; ++e) ov[4 + e] = __shfl_xor(ov[e], 16);   // next 4 columns (even lane groups)
                const bool writer = EPL == 8 ? (lgrp % 2) == 0 : true;
                if (live && writer)
                    put_operand_run<T>((T*)a.rn_hi, (T*)a.rn_lo, xfrag_elem<T>(m, col0, a.rn_MT), ov, H16);
                if (live && lgrp == 0) a.rsq[(size_t)nt * a.rsq_stride + m] = ss;
            }
        return;
    }
    if (a.sw_hi) {
        // SwiGLU: the lane's up values sit 32 lanes away (column + 8); lane
        // groups 0 and 1 form h for FFN columns 8 nt + 4 lgrp + e and one
        // lane writes each run of EPL consecutive columns, as the row kernel
        // does (same values, same arithmetic)
        constexpr int EPL = Elt<T>::EPL;
#pragma unroll
        for (int j = 0; j < WT; ++j)
#pragma unroll
            for (int i = 0; i < WT; ++i) {
                const int mt = mt0 + j, nt = nt0 + i, m = mt * 16 + lrow;
                const bool live = mt < a.MT && m < a.M && nt < a.n_tiles;
                const f32x4 v = acc[j][i] * s_rm[m - bm * BT * 16];
                float h[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float gt = v[e], up = __shfl_xor(v[e], 32);
                    h[e] = gt / (1.f + __expf(-gt)) * up;
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) h[4 + e] = __shfl_xor(h[e], 16);   // lane group 0 gets columns 4..7
                const bool writer = EPL == 8 ? lgrp == 0 : lgrp < 2;
                if (live && writer)
                    put_operand_run<T>((T*)a.sw_hi, (T*)a.sw_lo, xfrag_elem<T>(m, nt * 8 + lgrp * 4, a.sw_MT), h, H16);
            }
        return;
    }
#pragma unroll
    for (int j = 0; j < WT; ++j)
#pragma unroll
        for (int i = 0; i < WT; ++i) {
            const int mt = mt0 + j, nt = nt0 + i, m = mt * 16 + lrow;
            if (mt >= a.MT || m >= a.M || nt >= a.n_tiles) continue;
            const float rm = s_rm[m - bm * BT * 16];
            const f32x4 v = acc[j][i] * rm;
            *(float4*)(a.out + (size_t)blockIdx.z * a.out_kstride + (size_t)m * a.ldo + nt * 16 + lgrp * 4) =
                float4{v[0], v[1], v[2], v[3]};
        }
}



template <int WT>
static hipError_t launch_gemm_big_wt(int dtype, const BigGemmArgs& a, hipStream_t st) {
    const int gn = (a.n_tiles + 2 * WT - 1) / (2 * WT), gm = (a.MT + 2 * WT - 1) / (2 * WT);
    if ((a.m_fast ? gn : gm) > 65535) return hipErrorInvalidValue;     // grid y limit
    const int ks = a.kper > 0 ? (a.kb + a.kper - 1) / a.kper : 1;
    if (ks > 1 && (ks > BIG_KSPLIT_MAX || a.out_kstride < (size_t)a.M * a.ldo || !a.out || a.arg_val || a.sw_hi ||
                   a.rx || a.lrt > 0 || a.n_sq > 0))
        return hipErrorInvalidValue;
    const dim3 grid(a.m_fast ? gm : gn, a.m_fast ? gn : gm, ks), block(256);
    if (dtype == PBD_DTYPE_BF16) {
        if (a.op_f16) {
            if (a.xlo) return hipErrorInvalidValue;
            PBD_LAUNCH((k_gemm_big<bf16, false, WT, true>), grid, block, 0, st, a);
        } else {
            if (!a.xlo) return hipErrorInvalidValue;
            PBD_LAUNCH((k_gemm_big<bf16, true, WT, false>), grid, block, 0, st, a);
        }
    } else {
        if (a.op_f16) return hipErrorInvalidValue;
        PBD_LAUNCH((k_gemm_big<float, false, WT, false>), grid, block, 0, st, a);
    }
    return hipGetLastError();
}

// Sum of the K slices of a split-K large-M launch, in slice order:
// dst[i] = src[i] + src[stride + i] + ... (n a multiple of 4, 16-byte aligned)
__global__ __launch_bounds__(256) void k_ksum(KSumArgs a) {
    const size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (i >= a.n) return;
    float4 v = *(const float4*)(a.src + i);
    for (int s = 1; s < a.S; ++s) {
        const float4 w = *(const float4*)(a.src + (size_t)s * a.stride + i);
        v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    *(float4*)(a.dst + i) = v;
}

hipError_t launch_ksum(const KSumArgs& a, hipStream_t st) {
    if (a.n % 4 || a.stride % 4 || a.S < 1 || a.S > BIG_KSPLIT_MAX) return hipErrorInvalidValue;
    if (a.n == 0) return hipSuccess;
    PBD_LAUNCH(k_ksum, dim3((unsigned)((a.n / 4 + 255) / 256)), dim3(256), 0, st, a);
    return hipGetLastError();
}

// The tied LM head (argmax epilogue) takes 128 x 128 blocks (twice the MFMA
// work per byte of LDS traffic) when they still give every CU four
// work-groups and pad at most one row in eight; everything else takes
// 64 x 64, whose extra work-groups hide more latency (measured faster for
// the projections at up to 1056 rows)
hipError_t launch_gemm_big(int dtype, const BigGemmArgs& a, hipStream_t st) {
    if (!a.arg_val && !a.sw_hi && !a.rx && !a.out) return hipErrorInvalidValue;   // no destination
    const int bm8 = (a.MT + 7) / 8;
    const long big_blocks = (long)bm8 * ((a.n_tiles + 7) / 8);
    if (a.arg_val && big_blocks >= 4 * 256 && (bm8 * 8 - a.MT) * 8 <= a.MT) return launch_gemm_big_wt<4>(dtype, a, st);
    return launch_gemm_big_wt<2>(dtype, a, st);
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t st) {
    PBD_LAUNCH(k_accept, dim3((a.B + 63) / 64), dim3(64), 0, st, a);
    return hipGetLastError();
}
hipError_t launch_bf16_to_f16(const void* src, void* dst, size_t n_words, hipStream_t st) {
    PBD_LAUNCH(k_bf16_to_f16, dim3(1024), dim3(256), 0, st, (const uint32_t*)src, (uint32_t*)dst, n_words);
    return hipGetLastError();
}

hipError_t launch_fill_u32(void* p, size_t n_words, uint32_t v, hipStream_t st) {
    if (n_words == 0) return hipSuccess;
    PBD_LAUNCH(k_fill_u32, dim3(1024), dim3(256), 0, st, (uint32_t*)p, n_words, v);
    return hipGetLastError();
}

}  // namespace pbd
