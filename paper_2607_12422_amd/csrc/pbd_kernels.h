// Internal interface between the C-ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/pbd.h"

namespace pbd {

enum PassMode { PASS_DRAFT = 0, PASS_VERIFY = 1, PASS_PREFILL = 2 };
enum Epilogue { EPI_STORE = 0, EPI_PARTIAL = 1, EPI_SWIGLU = 2, EPI_ARGMAX = 3 };
enum TailMode { TAIL_SINGLE = 0, TAIL_BY_TILE = 1, TAIL_BY_ROW_HALF = 2 };
enum RowMap { MAP_CONCAT = 0, MAP_INTERLEAVE2 = 1 };

constexpr int MAX_NORM_DIM = 8192;     // hidden size bound for k_norm
constexpr int MAX_SHRINK_DIM = 8192;   // ffn and n_q*head_dim bound

struct AssembleArgs {
    int mode;
    int W, H, vocab, mask_id, max_seq;
    int chunk_pos, max_len;
    const int* seq_len;    // draft/verify: positions
    const int* anchor;
    const int* drafts;     // verify: [B][W-1]
    const int* prompt;     // prefill: [B][max_len]
    const int* lengths;    // prefill: [B]
    int* tokens;           // [B][W]
    int* pos0;             // [B]
    int* nrows;            // [B]
    int* status;
    const void* embed;     // packed [V/16][H/FK] fragments
    float* x;              // [M][H]
};

struct NormArgs {
    int M, MT, H;
    float eps;
    float* x;
    const float* partials;
    int n_partials;
    size_t partial_stride;  // floats between partial slabs
    const void* gain;
    void* xfrag;            // operand fragments, K = H
    void* xfrag_lo;         // bf16 residual of the operand (split operands) or null
    int n_src, r;
    float scale;
    const void* lora_a[3];  // [r][H]
    void* tail[3];          // tail operand fragments per source
};

struct ShrinkArgs {
    int M, MT, K, r;
    float scale;
    const void* xfrag;
    const void* xfrag_lo;   // or null
    const void* lora_a;     // [r][K]
    void* tail;
};

struct GemmArgs {
    const uint4* w;         // packed tiles: n_tiles x ft fragments
    int n_tiles, ft, kb, ks;
    int tail_frags, r, tail_mode, tile_split0, tile_split1;
    const uint4* x;         // operand fragments [kb][MT]
    const uint4* xlo;       // residual operand fragments (split operands) or null
    const uint4* xt[3];     // tail operand fragments [tail][MT]
    int M, MT;
    // epilogue
    float* out;             // STORE / PARTIAL
    int ldo;                // row stride of out / logits
    size_t partial_stride;
    void* out_frag;         // SWIGLU: down-projection operand
    void* out_frag_lo;      // SWIGLU: its residual fragments or null
    int out_MT;
    float* logits;          // ARGMAX: optional [M][V]
    float* arg_val;         // ARGMAX: [n_tiles][M]
    int* arg_idx;
    int exclude;            // ARGMAX: token id excluded (-1: none)
};

struct AttnArgs {
    int layer, max_batch, n_q, n_kv, nblk, W, G;
    int nqkv;
    int kps, s_launch;
    int causal, write_kv, qk_norm;
    float eps, scale_log2;
    size_t smem_main;
    const int* pos0;
    const int* nrows;
    const float* qkv;       // [M][nqkv] raw projections
    const void* q_norm;
    const void* k_norm;
    const float2* rope;     // [max_seq][head_dim/2] (cos, sin)
    void* kcache;           // [L][Bmax][n_kv][nblk][16*head_dim] fragment blocks
    void* vcache;
    float* part_o;          // [B][n_q][W][s_launch][head_dim]
    float* part_ml;         // [B][n_q][W][s_launch][2]
};

struct CombineArgs {
    int M, MT, W, n_q, head_dim, kps, s_launch, r;
    float scale;
    const int* pos0;
    const float* part_o;
    const float* part_ml;
    void* xfrag;
    void* xfrag_lo;
    const void* lora_a;     // [r][n_q*head_dim] or null
    void* tail;
};

struct ArgmaxArgs {
    int M, W, n_tiles, mode, chunk_pos;
    const float* arg_val;
    const int* arg_idx;
    int* out;
    const int* lengths;
    const int* nrows;
    int* seq_len_out;
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

struct PackArgs {
    int n_tiles, ft, kb, K, r, row_map, n_src;
    int src_rows[3];
    const void* w[3];
    const void* b[3];
    void* dst;
};

hipError_t launch_assemble(int dtype, const AssembleArgs& a, int batch, hipStream_t st);
hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t st);
hipError_t launch_shrink(int dtype, const ShrinkArgs& a, hipStream_t st);
hipError_t launch_gemm(int dtype, const GemmArgs& a, int epi, hipStream_t st);  // split iff a.xlo
hipError_t launch_attn(int dtype, int head_dim, int qt, const AttnArgs& a, int batch, hipStream_t st);
hipError_t launch_combine(int dtype, const CombineArgs& a, hipStream_t st);
hipError_t launch_argmax(const ArgmaxArgs& a, hipStream_t st);
hipError_t launch_accept(const AcceptArgs& a, hipStream_t st);
hipError_t launch_pack(int dtype, const PackArgs& a, hipStream_t st);
hipError_t launch_fill_u32(void* p, size_t n_words, uint32_t v, hipStream_t st);
size_t attn_smem_main(int dtype, int head_dim, int qt);
size_t attn_smem_bytes(int dtype, int head_dim, int qt);

}  // namespace pbd
