// Interface of the persistent batch-1 layer-stack kernel (pbd_fused.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/pbd.h"

namespace pbd {

constexpr int FUSED_MAX_ROWS = 32;     // block rows of one pass (B = 1, D + 1 <= 32)

struct FusedArgs {
    int L;                  // layers run (early-exit drafts: fewer than the model's)
    int M;                  // block rows (D + 1)
    int qk_norm;
    int full_from;          // block key i visible to block row j iff i <= j or j >= full_from
    int kv_rows;            // block rows whose K/V are appended to the cache (verify: M)
    int Bmax, nblk;         // KV-cache geometry
    int lm_MT;              // m-tiles of the LM-head operand
    int lm_sq_stride;
    unsigned spin_limit;    // polls before a wait gives up (PBD_STATUS_TIMEOUT)
    float eps, scale, scale_log2;
    const int* pos0;        // block start position (from the assembly kernel)
    const int* nrows;       // rows assembled (0: the sequence was skipped for capacity; nothing runs)
    int force_timeout;      // tests: every work-group first waits on a word no one sets
    const float* x0;        // assembled residual [M][hidden]
    const void* pk;         // packed weights
    // byte offsets into the packed weights (below 4 GiB; checked by the caller)
    uint32_t lay_stride;    // between consecutive layers' packed blocks
    uint32_t off_qkv, off_o, off_gu, off_d, off_attn_norm, off_mlp_norm, off_q_norm, off_k_norm;   // layer 0
    uint32_t off_la[7];
    uint32_t off_lb_qkv, off_lb_o, off_lb_gu, off_lb_d;
    const void* final_norm;
    const float2* rope;
    char* kcache;
    char* vcache;
    void* ws;               // the kernel's own workspace region (fused_ws_bytes())
    void* lm_hi;            // LM-head operand fragments (value, residual) and row sums of squares
    void* lm_lo;
    float* lm_sq;
    int* status;
};

size_t fused_ws_bytes();
size_t fused_lds_bytes();
int fused_threads();
// control words of the region: [0, 8) per-XCD rank tickets, [8] epoch, [9] abort
size_t fused_ctl_offset();
// stage timestamps [8 groups][32 ranks][64 layers][8 stages][4] (uint64,
// 100 MHz): when the stage's wait began, when its inputs were ready, when
// its compute waves finished (GEMM stages) and when its output was published;
// layer L holds the final stage's start and end (stage 0, points 0 and 1)
size_t fused_trace_offset();
int fused_trace_entries();
// resident work-groups per CU of the kernel (sets its dynamic-LDS limit first)
hipError_t fused_occupancy(int* blocks_per_cu);
hipError_t launch_fused(const FusedArgs& a, bool lora, hipStream_t st);

}  // namespace pbd
