// Internal interface between the C-ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/pbd.h"

namespace pbd {

enum PassMode { PASS_DRAFT = 0, PASS_VERIFY = 1, PASS_PREFILL = 2 };
// GEMM epilogues: raw q/k/v; residual add + next RMSNorm operand; SwiGLU; LM head argmax
enum Epilogue { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_ARGMAX = 3 };
// which LoRA shrink matrix a GEMM tile uses
enum LoraMode { LORA_SINGLE = 0, LORA_BY_TILE = 1, LORA_ROW_HALF = 2 };
enum RowMap { MAP_CONCAT = 0, MAP_INTERLEAVE2 = 1 };

constexpr int MAX_RT = 4;              // LoRA rank <= 64: up to four 16-row shrink tiles
constexpr int KSPLIT_MAX = 4;          // K slices of a split-K GEMM

struct AssembleArgs {
    int mode;
    int W, H, vocab, mask_id, max_seq;
    int chunk_pos, max_len, MT, m_stride;
    int lead;              // draft/verify: leading anchor rows (1, or 0 for a block of drafts only)
    int room;              // prefill: rows a prompt must leave free in the cache (D + 1)
    int pos_add;           // draft/verify: the block starts at seq_len + pos_add
    const int* seq_len;    // draft/verify: positions
    const int* anchor;
    const int* drafts;     // verify: [B][W-lead]; draft: null (all masks) or the partly denoised block
    const int* prompt;     // prefill: [B][max_len]
    const int* lengths;    // prefill: [B]
    int* tokens;           // [B][W]
    int* pos0;             // [B]
    int* nrows;            // [B]
    int* status;
    const void* embed;     // packed [V/16][H/FK] fragments
    const void* gain;      // attention RMSNorm gain of layer 0
    float* x;              // [M][H] residual
    void* op_hi;           // first QKV operand x*g (fragments) and its bf16 residual
    void* op_lo;
    int op_f16;            // bf16 model: the operand as fp16 in op_hi (op_lo unused)
    float* sq;             // [1][m_stride] per-row sum of squares
    unsigned* fused_ctl;   // persistent pass next: its rank tickets and abort word are cleared and its epoch advanced (null: none)
    int fused_layers;      // layers that pass runs (it advances the per-parity write counts of its partial buffers)
};

struct FGemmArgs {
    const uint4* w;         // weight tiles: [n_tiles][kb] fragments
    int n_tiles, kb;
    const uint4* xhi;       // operand fragments [kb][MT]
    const uint4* xlo;       // operand residual fragments or null
    int M, MT;
    // RMSNorm folded in: r_m = rsqrt(sum_p sq[p*sq_stride + m] / norm_dim + eps); n_sq = 0: r_m = 1
    const float* sq;
    int n_sq, sq_stride, norm_dim;
    float eps;
    // rows per sequence; block rows j = m % W below adapter_from run without
    // the adapter, and below excl_from without the argmax exclusion
    int W, adapter_from, excl_from;
    // LoRA: shrink u = s * r_m * A x in the tile, expand B u
    int lora, rt, lora_mode, tile_split0, tile_split1;
    float scale;
    const uint4* la[3];     // shrink tiles per source: [rt][kb] fragments
    const void* lb;         // expand blocks: [n_tiles][rt] x 64 lanes x 4 elements
    // epilogues
    float* out;             // STORE: [M][ldo]
    int ldo;
    float* x;               // RESID: residual [M][ldx]
    int ldx;
    const void* gnext;      // RESID: gain of the next RMSNorm
    void* nx_hi;            // RESID: next operand fragments (K = ldx) / SWIGLU: h fragments
    void* nx_lo;
    int n_MT;
    float* sq_out;          // RESID: [n_tiles][sq_stride] per-tile row sums of squares
    float* logits;          // ARGMAX: optional [M][ldo]
    float* arg_val;         // ARGMAX: [n_tiles][M]
    int* arg_idx;
    int exclude;            // ARGMAX: token id excluded (-1: none)
    // ARGMAX with confidence (null: none): per partial, the row's maximum over
    // all columns and the sum of exp(value - that maximum), same layout as arg_val
    float* arg_mx;
    float* arg_sum;
    // split-K (ksplit > 1: one m-group only): partial tiles [n_tiles][ksplit][MG*256]
    // and per-tile arrival counters (zero between launches)
    int ksplit;
    float* part;
    unsigned* cnt;
};

struct AttnArgs {
    int layer, max_batch, n_q, n_kv, nblk, W, G;
    int nqkv;
    int kps, s_launch;
    int n_qgrp;             // work-groups per (split, KV head, sequence), each over QT query tiles
    // block key i is visible to block row j iff i <= j or j >= full_from
    // (full_from = W: causal; 0: bidirectional); rows j < kv_rows append their K/V
    int full_from, kv_rows, qk_norm;
    float eps, scale_log2;
    size_t smem_main;
    const int* pos0;
    const int* nrows;
    const float* qkv;       // [M][nqkv] projections
    const void* q_norm;
    const void* k_norm;
    const float2* rope;     // [max_seq][head_dim/2] (cos, sin)
    void* kcache;           // [L][Bmax][n_kv][nblk][16*head_dim] fragment blocks
    void* vcache;
    float* part_o;          // [B][n_q][W][s_launch][head_dim]
    float* part_ml;         // [B][n_q][W][s_launch][2]
    // pf_x extra grid columns of work-groups touch the ranges [pf[i],
    // pf[i] + pf_bytes[i]) once per 128-byte line (at most 16 lines per
    // thread), warming the memory-side cache for the kernels that follow
    int pf_x;
    const char* pf[3];
    size_t pf_bytes[3];
    // chunk mode (prefill): the W block rows' K/V are already in the cache at
    // positions t..t+nrows-1; every key is read from the cache, causal inside
    // the chunk; no block split and no K/V writes
    int chunk;
    // every split is run by k_attn_rows (launch_attn_rows); k_attn only warms
    // the memory-side cache in its pf_x extra columns
    int skip_prefix;
};

// Prefill chunk K/V: norm + RoPE of the W rows' keys, appended with the values.
struct KVWriteArgs {
    int layer, max_batch, n_q, n_kv, nblk, W, nqkv, qk_norm;
    float eps;
    const int* pos0;
    const int* nrows;
    const float* qkv;       // [M][nqkv] projections
    const void* k_norm;
    const float2* rope;
    void* kcache;
    void* vcache;
};

// Prefill: each sequence's last prompt row of the chunk (final-norm operand
// fragments and row sum-of-squares partials) gathered into row b of a compact
// operand, so the LM head runs on batch rows only.
struct GatherArgs {
    int W, MT, MTc, kb, n_sq, sq_stride, sqc_stride, chunk_pos;
    const int* lengths;
    const int* nrows;
    const void* x_hi;       // operand fragments [kb][MT]
    const void* x_lo;
    const float* sq;        // [n_sq][sq_stride]
    void* c_hi;             // compact operand fragments [kb][MTc]
    void* c_lo;
    float* c_sq;            // [n_sq][sqc_stride]
};

// Large-M projection (prefill chunks): out[m][16 t + r] = r_m * (W x_m)[16 t + r]
// for every row m and weight tile t, on the same packed operands as FGemmArgs.
constexpr int BIG_KSPLIT_MAX = 8;     // K slices of a split-K large-M launch

struct BigGemmArgs {
    const uint4* w;         // weight tiles [n_tiles][kb] fragments
    int n_tiles, kb;
    const uint4* xhi;       // operand fragments [kb][MT]
    const uint4* xlo;       // residual fragments or null
    int M, MT;
    const float* sq;        // RMSNorm partials [n_sq][sq_stride]; n_sq = 0: r_m = 1
    int n_sq, sq_stride, norm_dim;
    float eps;
    float* out;             // [M][ldo] fp32
    int ldo;
    // LoRA expand (lrt > 0), added before the r_m scaling: acc += s * B u, with
    // u [M][ldu] fp32 the shrink A x of source sc at columns sc * lrt * 16, B
    // blocks [n_tiles][lrt] x 64 lanes x 4 elements; the source of a tile is
    // chosen as in the small-M GEMM (lora_mode, tile_split0/1); block rows
    // m % W < adapter_from take no adapter
    const float* u;
    int ldu, lrt, lora_mode, tile_split0, tile_split1, W, adapter_from;
    float scale;
    const void* lb;
    // argmax epilogue (arg_val set; tied LM head): per 16-column tile and row
    // the (max, argmax) with column `exclude` skipped on block rows m % W >=
    // excl_from, ties to the lowest column, into arg_val/arg_idx [n_tiles][M];
    // optional logits [M][ldo] and softmax partials arg_mx/arg_sum (maximum
    // over the tile and sum of exp(value - maximum)); out is not written
    float* logits;
    float* arg_val;
    int* arg_idx;
    float* arg_mx;
    float* arg_sum;
    int exclude, excl_from;
    // grid order: m-blocks fastest (the blocks that share weight tiles run
    // together; for weights larger than the memory-side cache)
    int m_fast;
    // split-K (plain STORE epilogue, no RMSNorm; the LoRA shrink): grid z =
    // ceil(kb / kper) slices of kper K fragments (kper = 0: one slice); slice
    // z stores its products at out + z * out_kstride, summed afterwards by
    // launch_ksum
    int kper;
    size_t out_kstride;     // floats, >= M * ldo
    // SwiGLU epilogue (sw_hi set; gate/up tiles with rows 0-7 gate and 8-15
    // up of the same FFN columns): h = silu(gate) * up written as the down
    // projection's operand fragments (K = n_tiles * 8, sw_MT m-tiles); out is
    // not written
    void* sw_hi;
    void* sw_lo;
    int sw_MT;
    // residual epilogue (rx set; n = hidden): x += y in place ([M][ldx]
    // fp32), the next RMSNorm operand x * rgain as fragments (rn_MT m-tiles)
    // and the tile's row sums of squares rsq[tile * rsq_stride + m]; out is
    // not written
    float* rx;
    int ldx;
    const void* rgain;
    void* rn_hi;
    void* rn_lo;
    int rn_MT;
    float* rsq;
    int rsq_stride;
    // bf16 model, single fp16 operands: xhi holds fp16 fragments (xlo null),
    // w points to fp16 copies of the weight fragments, and the residual /
    // SwiGLU epilogues write fp16 operands (rn_lo / sw_lo unused)
    int op_f16;
};

struct CombineArgs {
    int W, n_q, head_dim, kps, s_launch, MT;
    int M;                  // block rows of the pass (set by launch_combine)
    const int* pos0;
    const float* part_o;
    const float* part_ml;
    void* op_hi;            // O-projection operand fragments (K = n_q*head_dim)
    void* op_lo;
    int op_f16;             // bf16 model: the operand as fp16 in op_hi (op_lo unused)
};

struct ArgmaxArgs {
    int M, W, n_tiles, mode, chunk_pos;
    int lead;               // draft: rows j >= lead are draft rows, out[b][j - lead]
    int* out0;              // draft: argmax of row 0 when lead = 1 (null: dropped), at out0[b * out0_stride]
    int out0_stride;
    int out_stride, out_off;  // verify: out[b * out_stride + out_off + j]
    int compact;            // prefill: row m is sequence m's last prompt row (gathered), if in this chunk
    const float* arg_val;
    const int* arg_idx;
    int* out;
    const int* lengths;
    const int* nrows;
    int* seq_len_out;
    // draft with confidence (null: none): the log-probability of each row's
    // argmax under the softmax of the whole row, [B][W-1] like out
    const float* arg_mx;
    const float* arg_sum;
    float* conf;
};

// One remasking pass of multi-step denoising: among the still-masked positions
// of each sequence (block entry == mask id), fix the n_fix whose candidate has
// the highest confidence (equal confidences: lower position first).
struct RemaskArgs {
    int D, mask_id, n_fix, step;
    const int* cand;        // [B][D] candidates of this pass
    const float* cand_conf; // [B][D] their confidences
    int* block;             // [B][D] block state, updated in place
    float* conf;            // optional [B][D]: confidence at which a position was fixed
    int* fixed_at;          // optional [B][D]: pass (1-based) that fixed it
};

struct AcceptArgs {
    int B, D, max_seq;
    const int* draft;
    const int* verify;
    const int* forced;
    int* seq_len;
    int* anchor;
    int* n_acc;
    int* out;
    int* status;
};

// Repack row-major matrices into fragment tiles (W and LoRA shrink A).  Rows
// past `rows_total` are zero.
struct PackArgs {
    int n_tiles, kb, K, row_map, n_src, rows_total;
    int src_rows[3];
    const void* w[3];
    void* dst;
};

// Repack LoRA B [rows][r] into expand blocks of the GEMM output tiles.
struct PackExpandArgs {
    int n_tiles, rt, r, row_map, n_src;
    int src_rows[3];
    const void* b[3];
    void* dst;
};

hipError_t launch_assemble(int dtype, const AssembleArgs& a, int batch, hipStream_t st);
hipError_t launch_fgemm(int dtype, const FGemmArgs& a, int epi, hipStream_t st);   // split iff a.xlo
int fgemm_mgroup(int epi, int MT, int lrt);   // lrt: LoRA rank tiles of the launch (0: adapter off)
int fgemm_threads(int epi);         // work-group size of the GEMM with epilogue epi
// The attention partials of a draft or verify pass with four or five 16-row
// query tiles per KV head (bf16, head_dim 128, W <= 48): every split of
// k_attn's schedule, one wave per query tile, keys staged through LDS
// (false: this shape is not covered; use k_attn alone)
bool attn_rows_fits(int dtype, int head_dim, int qt, int chunk, int W);
hipError_t launch_attn_rows(const AttnArgs& a, int qt, int batch, hipStream_t st);
hipError_t launch_attn(int dtype, int head_dim, int qt, const AttnArgs& a, int batch, hipStream_t st);
hipError_t launch_combine(int dtype, const CombineArgs& a, int M, hipStream_t st);
hipError_t launch_argmax(const ArgmaxArgs& a, hipStream_t st);
// persistent LM head: `grid` work-groups, one (max, argmax) partial each per row
// (and one softmax partial when a.arg_sum is set)
bool lmhead_fits(int kb, int MT);
hipError_t launch_lmhead(int dtype, const FGemmArgs& a, int grid, hipStream_t st);
hipError_t launch_accept(const AcceptArgs& a, hipStream_t st);
hipError_t launch_kvwrite(int dtype, int head_dim, const KVWriteArgs& a, int batch, hipStream_t st);
hipError_t launch_gather_last(int dtype, const GatherArgs& a, int batch, hipStream_t st);
// dst[i] = sum over s < S of src[s * stride + i] in slice order (the K
// slices of a split-K large-M launch); n and stride multiples of 4
struct KSumArgs {
    float* dst;
    const float* src;
    size_t n, stride;
    int S;
};
hipError_t launch_ksum(const KSumArgs& a, hipStream_t st);
hipError_t launch_gemm_big(int dtype, const BigGemmArgs& a, hipStream_t st);   // split iff a.xlo
hipError_t launch_remask(const RemaskArgs& a, int batch, hipStream_t st);
hipError_t launch_pack(int dtype, const PackArgs& a, hipStream_t st);
hipError_t launch_pack_expand(int dtype, const PackExpandArgs& a, hipStream_t st);
hipError_t launch_fill_u32(void* p, size_t n_words, uint32_t v, hipStream_t st);
// fp16 copy of n_words words of packed bf16 pairs
hipError_t launch_bf16_to_f16(const void* src, void* dst, size_t n_words, hipStream_t st);
// profiling: events that the next launch records its start and end into (null: none)
void set_launch_events(hipEvent_t start, hipEvent_t stop);
void get_launch_events(hipEvent_t* start, hipEvent_t* stop);
size_t attn_smem_main(int dtype, int head_dim, int qt);
size_t attn_smem_bytes(int dtype, int head_dim, int qt);

}  // namespace pbd
