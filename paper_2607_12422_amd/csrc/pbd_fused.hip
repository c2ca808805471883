// Persistent single-launch layer stack of one batch-1 pass (draft or verify,
// Sec. 3 steps 1-3) for the Qwen3-0.6B layer shape on gfx950.
//
// Why one launch: at batch 1 a pass streams 0.9 GB of layer weights through
// 28 x 5 dependent stages.  As separate kernels each stage is a cold burst
// of 4-12 MB behind a launch, and the chain runs at about an eighth of the
// HBM rate.  Weights do not depend on activations, so a resident kernel can
// stream them continuously while the activations hop from stage to stage.
//
// Layout of the work (256 work-groups, one per CU, eight XCDs of 32):
//   * XCD g is "group" g and owns KV head g (the shape has exactly eight):
//     the q rows of heads 2g, 2g+1 and the k/v rows of head g, the attention
//     of that head, the O-projection K-slice of those two heads, and the
//     FFN columns [384 g, 384 g + 384) of gate/up and the matching K-slice of
//     down.  Every group keeps its own copy of the residual stream.
//   * Inside a group, rank r (0..31) owns the columns [32 r, 32 r + 32) of
//     the residual copy.
//   * Per layer: R (residual update from the eight groups' down-projection
//     partials, attention RMSNorm operand), Q (q/k/v tile), A (split-KV
//     attention partial), M (merge of the partials, one query row per rank),
//     O (O-projection partial over the group's heads), R2 (residual update
//     from the O partials, MLP RMSNorm operand), GU (gate/up tiles + SwiGLU),
//     D (down-projection partial over the group's FFN slice).
//   * Handoffs inside a group go through the XCD's L2: plain stores, then a
//     per-rank flag; consumers poll the flags and read with L1-bypassing
//     (sc1) loads.  Flags hold (epoch, layer).  The two handoffs between
//     groups per layer (O and down partials) are fp32 values written through
//     to memory whose lowest mantissa bit is a tag: the parity of the number
//     of writes that half of the buffer has received (counted on the device
//     across passes), so stale contents always carry the other bit and
//     consumers poll the data itself.  No fence is ever needed.  Buffers
//     alternate by layer parity.
//   * Each work-group has 8 compute waves and 2 loader waves.  The loader
//     waves stream the work-group's weight fragments and its attention
//     split's K/V blocks, in stage order, straight into an LDS ring with
//     global_load_lds (non-temporal), keeping up to the ring's 80 KiB in
//     flight.  Compute waves never issue a global load that a later wait
//     would have to drain behind the prefetch.  Loader waves take part in
//     every work-group barrier and wait for a stage's fragments before the
//     barrier that opens that stage.
//   * Every wait is bounded: on expiry the wait sets PBD_STATUS_TIMEOUT and
//     an abort word that releases every other waiter, and the kernel runs
//     to its end.
// RMSNorm is folded as in the skinny GEMM: operands carry x * g, per-rank
// row sums of squares give r_m, applied to the accumulators.  LoRA (App.
// A.2) runs unmerged in every tile (shrink on the same operand fragments,
// expand per wave before the cross-wave reduction; for the K-split O and
// down projections each group's partial carries its own expand, summed
// with the partials by linearity).
#include "pbd_device.h"
#include "pbd_fused.h"
#include "pbd_kernels.h"

#include <hip/hip_ext.h>

namespace pbd {
namespace fz {

constexpr int H = 1024, F = 3072, NQ = 16, NKV = 8, HD = 128, G = NQ / NKV;
constexpr int NGRP = 8, NRANK = 32;
constexpr int NWC = 6, NWL = 2, NTHR = (NWC + NWL) * WAVE;   // 8 waves: 256 VGPRs each
constexpr int MW = FUSED_MAX_ROWS;     // rows per pass
constexpr int QRMAX = G * MW;          // query rows per KV head
constexpr int KBH = H / 32;            // fragments over the hidden size
constexpr int FPW = (KBH + NWC - 1) / NWC;  // hidden-size fragments per compute wave (6)
constexpr int RR = NWC * WAVE / 16;   // rows per round of the residual stage (16 column pairs per row)
constexpr int NRR = (MW + RR - 1) / RR; // rounds
constexpr int KB_O = NQ * HD / 32;     // 64
constexpr int KB_D = F / 32;           // 96
constexpr int GQKV = (G + 2) * HD;     // a group's q/k/v columns (512)
constexpr int GO = G * HD;             // a group's O-projection K-slice (256)
constexpr int GF = F / NGRP;           // a group's FFN columns (384)
constexpr int NSLOT = 88;              // LDS ring slots of 1 KiB (even: the two loaders take alternate items)
static_assert(NSLOT % 2 == 0, "ring slots come in pairs");
constexpr int LOOKAHEAD = 12;          // ring items issued ahead per barrier interval (even)
constexpr int LDQ = HD + 8;            // bf16 row pitch of the attention LDS rows
constexpr int PB = HD + 4;             // fp32 pitch of a merged attention row
constexpr int APW = HD + 4;            // fp32 words per stored attention partial row (m, l, o[128], pad)

enum { ST_R = 0, ST_Q, ST_A, ST_M, ST_O, ST_R2, ST_GU, ST_D, NSTAGE };
enum { FL_R = 0, FL_Q, FL_A, FL_M, FL_R2, FL_GU, NFLAG };
constexpr int TRACE_LAYERS = 64;       // layers covered by the stage timestamps
// work-group barriers per stage (the loader waves take part in every one)
__host__ __device__ constexpr int n_barriers(int st) {
    return st == ST_A ? 4 : (st == ST_R || st == ST_M || st == ST_R2) ? 1 : 2;
}

// LDS map (bytes)
constexpr size_t RING_BYTES = (size_t)NSLOT * 1024;
constexpr size_t SRED_BYTES = (size_t)2 * NWC * 2 * WAVE * 16;                     // GEMM reduction
constexpr size_t QL_BYTES = (size_t)QRMAX * LDQ * 2, KL_BYTES = (size_t)32 * LDQ * 2, VL_BYTES = (size_t)32 * HD * 2;
constexpr size_t PBUF_BYTES = (size_t)4 * 16 * PB * 4;
constexpr size_t ATT_BYTES = QL_BYTES + KL_BYTES + VL_BYTES + PBUF_BYTES;
constexpr size_t SCR_BYTES = (SRED_BYTES > ATT_BYTES ? SRED_BYTES : ATT_BYTES);
constexpr size_t XS_BYTES = (size_t)MW * 32 * 4;
constexpr size_t MISC_BYTES = 512;
constexpr size_t LDS_BYTES = RING_BYTES + SCR_BYTES + XS_BYTES + MISC_BYTES;
static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");

// Workspace of the persistent pass (bytes), parity-doubled per-group buffers.
struct WsMap {
    size_t flags, xn, xm, sq, sqm, qkv, apart, oop, hop, parto, partd, ctl, trace, total;
};
__host__ __device__ inline WsMap ws_map() {
    WsMap w{};
    size_t off = 0;
    auto take = [&](size_t b) { size_t o = off; off += (b + 255) / 256 * 256; return o; };
    w.flags = take((size_t)NFLAG * 2 * NGRP * NRANK * 4);
    w.xn = take((size_t)2 * NGRP * MW * H * 4);
    w.xm = take((size_t)2 * NGRP * MW * H * 4);
    w.sq = take((size_t)2 * NGRP * NRANK * MW * 4);
    w.sqm = take((size_t)2 * NGRP * NRANK * MW * 4);
    w.qkv = take((size_t)2 * NGRP * MW * GQKV * 4);
    w.apart = take((size_t)2 * NGRP * NRANK * QRMAX * APW * 4);
    w.oop = take((size_t)2 * NGRP * MW * GO * 4);
    w.hop = take((size_t)2 * NGRP * MW * GF * 4);
    w.parto = take((size_t)2 * NGRP * MW * H * 4);
    w.partd = take((size_t)2 * NGRP * MW * H * 4);
    w.ctl = take(256);
    w.trace = take((size_t)NGRP * NRANK * TRACE_LAYERS * NSTAGE * 4 * 8);
    w.total = off;
    return w;
}

typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned u32x2;

// Cache-policy bits of buffer instructions: sc0 = 1, nt = 2, sc1 = 16.
constexpr int SC1 = 16, SC01 = 17, NT = 2;
// Range of the workspace's buffer resource (bytes).
constexpr unsigned WS_RANGE = 0x7fffffffu;

__device__ __forceinline__ unsigned xcc_id() {
    unsigned v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 16)" : "=s"(v));
    return v & 0xf;
}

__device__ __forceinline__ unsigned ld_sc1_u32(const unsigned* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until vmcnt <= n for a run-time n in [0, 40] (loader waves).
__device__ __forceinline__ void wait_vm(int n) {
#define PBD_VMW(k) case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
    switch (n) {
        PBD_VMW(0) PBD_VMW(1) PBD_VMW(2) PBD_VMW(3) PBD_VMW(4) PBD_VMW(5) PBD_VMW(6) PBD_VMW(7)
        PBD_VMW(8) PBD_VMW(9) PBD_VMW(10) PBD_VMW(11) PBD_VMW(12) PBD_VMW(13) PBD_VMW(14) PBD_VMW(15)
        PBD_VMW(16) PBD_VMW(17) PBD_VMW(18) PBD_VMW(19) PBD_VMW(20) PBD_VMW(21) PBD_VMW(22) PBD_VMW(23)
        PBD_VMW(24) PBD_VMW(25) PBD_VMW(26) PBD_VMW(27) PBD_VMW(28) PBD_VMW(29) PBD_VMW(30) PBD_VMW(31)
        PBD_VMW(32) PBD_VMW(33) PBD_VMW(34) PBD_VMW(35) PBD_VMW(36) PBD_VMW(37) PBD_VMW(38) PBD_VMW(39)
        default: asm volatile("s_waitcnt vmcnt(40)" ::: "memory"); break;
    }
#undef PBD_VMW
}

__device__ __forceinline__ void bar() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// LoRA expand acc += B u over the adapter's 16 rank entries: the bf16 B block
// (lane: output row lane % 16, rank entries 4 (lane / 16) ..) and the scaled
// shrink u (the shrink accumulator's layout) both as fp16 operands
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4;
__device__ __forceinline__ void mma_k4h(f32x4& acc, const uint2& a, const f32x4& p) {
    f16x4 av, pv;
    const unsigned u[2] = {a.x, a.y};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        av[2 * i] = (_Float16)__uint_as_float(u[i] << 16);
        av[2 * i + 1] = (_Float16)__uint_as_float(u[i] & 0xffff0000u);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) pv[e] = (_Float16)p[e];
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(av, pv, acc, 0, 0, 0);
}

// The layer GEMMs feed the matrix cores fp16 operands: the activations are
// stored as fp16 (11 significant bits), and the projection and LoRA A
// fragments are read from an fp16 copy of the packed bf16 weights made at
// initialisation.  A bf16 value of magnitude in [2^-14, 65504] is exactly an
// fp16 value; smaller weights round to the fp16 subnormal grid (absolute
// error below 2^-25).
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
__device__ __forceinline__ f16x8 w_f16(const uint4& w) { return __builtin_bit_cast(f16x8, w); }
// acc += W_frag * X_frag (the activation fragment holds fp16 values)
__device__ __forceinline__ void mma_h(f32x4& acc, const f16x8& w, const uint4& x) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(w, __builtin_bit_cast(f16x8, x), acc, 0, 0, 0);
}
__device__ __forceinline__ unsigned f16_pair(float a, float b) {
    return (unsigned)__builtin_bit_cast(unsigned short, (_Float16)a) |
           ((unsigned)__builtin_bit_cast(unsigned short, (_Float16)b) << 16);
}

// Byte offset of element (row m, column k) of a fragment-major fp16
// activation operand: fragment k / 32 of m-tile m / 16 is 1 KiB at
// (2 (k / 32) + m / 16) * 1024, in MFMA operand order (lane = 16 k-group +
// row, eight consecutive k per lane).
__device__ __forceinline__ unsigned opnd_elem(int m, int k) {
    return (unsigned)(((((k / 32) * 2 + m / 16) * 64 + ((k % 32) / 8) * 16 + m % 16) * 8 + k % 8) * 2);
}

// Static per-work-group schedule: which weight tiles, K/V blocks and
// fragments a rank loads in each stage.
struct Sched {
    int g, r, t, nkb, s_pre;
    // Q tile (global tile index in the packed q/k/v weights) of this rank
    __device__ __forceinline__ int q_tile() const { return r < 16 ? 16 * g + r : (r < 24 ? 128 + 8 * g + (r - 16) : 192 + 8 * g + (r - 24)); }
    // LoRA source of the Q tile: 0 q, 1 k, 2 v
    __device__ __forceinline__ int q_src() const { return r < 16 ? 0 : (r < 24 ? 1 : 2); }
    __device__ __forceinline__ int gu_t1() const { return 48 * g + r; }
    __device__ __forceinline__ int gu_t2() const { return 48 * g + 32 + r / 2; }
    // prefix key blocks of this rank's attention split (rank 31: the block keys)
    __device__ __forceinline__ int kb_begin() const { return r < s_pre ? (r * nkb) / s_pre : 0; }
    __device__ __forceinline__ int kb_count() const { return r < s_pre ? ((r + 1) * nkb) / s_pre - (r * nkb) / s_pre : 0; }
    __device__ __forceinline__ int items(int st) const {
        switch (st) {
            case ST_Q: return KBH;
            case ST_A: return 8 * kb_count();
            case ST_O: return 16;
            case ST_GU: return 2 * KBH;
            case ST_D: return 24;
            default: return 0;
        }
    }
};

template <bool LORA>
__global__ __launch_bounds__(NTHR, 1) void k_fused(FusedArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* ring = smem;
    unsigned char* scr = smem + RING_BYTES;
    float* xs = (float*)(smem + RING_BYTES + SCR_BYTES);               // [MW][32] residual slice
    float* s_rm = (float*)(smem + RING_BYTES + SCR_BYTES + XS_BYTES);  // [MW]
    int* s_id = (int*)(s_rm + MW);                                       // group, rank, t
    unsigned* s_pub = (unsigned*)(s_id + 8);                             // waves past their stores

    int tid = threadIdx.x;
    const int wid = __builtin_amdgcn_readfirstlane(tid / WAVE);   // wave-uniform (scalar)
    int lane = tid % WAVE;
    int lrow = lane % 16, lgrp = lane / 16;
    const WsMap wm = ws_map();
    char* ws = (char*)a.ws;
    unsigned* ctl = (unsigned*)(ws + wm.ctl);
    unsigned* abort_w = ctl + 9;

    if (tid == 0) {
        const unsigned x = xcc_id();
        const unsigned rk = __hip_atomic_fetch_add(ctl + x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_id[0] = (int)x;
        s_id[1] = (int)rk;
        s_id[2] = a.pos0[0];
        s_id[3] = (int)ctl[8];
        s_id[4] = a.nrows[0];
        s_id[5] = (int)ctl[14];      // writes into the partial buffers' even / odd halves before this pass
        s_id[6] = (int)ctl[15];
        *s_pub = 0u;
    }
    __syncthreads();
    // a sequence skipped for capacity: no cache write, no outputs (every
    // work-group reads the same word, so all leave together)
    if (__builtin_amdgcn_readfirstlane(s_id[4]) == 0) return;
    // wave-uniform from here on (scalar registers, and so every address derived from them)
    Sched sc;
    sc.g = __builtin_amdgcn_readfirstlane(s_id[0]);
    sc.r = __builtin_amdgcn_readfirstlane(s_id[1]);
    sc.t = __builtin_amdgcn_readfirstlane(s_id[2]);
    const unsigned epoch = (unsigned)__builtin_amdgcn_readfirstlane(s_id[3]);
    const unsigned wbase0 = (unsigned)__builtin_amdgcn_readfirstlane(s_id[5]);
    const unsigned wbase1 = (unsigned)__builtin_amdgcn_readfirstlane(s_id[6]);
    // tag bit of the partials written at layer l: parity of that buffer half's write count
    auto ptag_bit = [&](int l) -> unsigned { return ((l & 1 ? wbase1 : wbase0) + (unsigned)(l >> 1) + 1u) & 1u; };
    if (sc.g >= NGRP || sc.r >= NRANK) {
        // placement is not 8 x 32 (never seen): report; the work-groups that
        // wait for the missing ranks time out and the pass ends with an error
        if (tid == 0) {
            atomicOr(a.status, PBD_STATUS_TIMEOUT);
            __hip_atomic_store(abort_w, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        return;
    }
    sc.nkb = (sc.t + 15) / 16;
    sc.s_pre = sc.nkb < NRANK - 1 ? sc.nkb : NRANK - 1;
    const int g = sc.g, r = sc.r, t = sc.t, M = a.M;
    const int QR = G * M, QT = (QR + 15) / 16;
    const int L = a.L;

    __amdgpu_buffer_rsrc_t rws = __builtin_amdgcn_make_buffer_rsrc(ws, 0, WS_RANGE, 0x00020000);

    // ------------------------------------------------------------------
    // Loader waves: ring fill in stage order, in step with the barriers.
    // ------------------------------------------------------------------
    if (wid >= NWC) {
        const int lid = wid - NWC;
        const char* pk = (const char*)a.pk;
        // Every stage's items are runs of consecutive 1 KiB fragments in
        // memory; item i is fragment i % per of run i / per, and run j starts
        // at base + (j & 1) * odd + (j >> 1) * pair (+ the layer's offset).
        // Stage sizes and run lengths are even, so with items dealt out by
        // the parity of their global index this loader takes offsets
        // lid, lid + 2, ... of every run.
        const int q_tile = sc.q_tile(), t1 = sc.gu_t1(), t2 = sc.gu_t2(), kb0 = sc.kb_begin();
        const bool half_mine = ((lrow / 4) & 1) == (r & 1);   // rows of the half gate/up tile
        const size_t kv_layer = (size_t)a.Bmax * NKV * a.nblk * 16 * HD * 2;
        const char* kv_k = a.kcache + (size_t)g * a.nblk * 16 * HD * 2 + (size_t)kb0 * (16 * HD * 2);
        const char* kv_v = a.vcache + (size_t)g * a.nblk * 16 * HD * 2 + (size_t)kb0 * (16 * HD * 2);
        // issue cursor: layer, stage, item (even), global item index, ring slot,
        // run, offset in the run, and the stage's run parameters
        int cl = 0, cs = -1, ci = 0, cn = 0, cg = 0, slot = 0, rj = 0, rk = 0;
        int per = 1;
        bool half = false;
        const char* sbase = pk;      // run 0 of the stage at layer cl
        const char* rbase = pk;      // current run
        long odd = 0, pair = 0;
        auto run_base = [&]() { rbase = sbase + (rj & 1) * odd + (rj >> 1) * pair; };
        auto enter_stage = [&]() {
            // stage cs of layer cl
            ci = 0; rj = 0; rk = 0;
            cn = sc.items(cs);
            half = false; odd = 0; pair = 0; per = 2;
            const char* lb = pk + (size_t)cl * a.lay_stride;
            switch (cs) {
                case ST_Q: per = KBH; sbase = lb + a.off_qkv + (size_t)q_tile * KBH * 1024; break;
                case ST_A:
                    per = 4; sbase = kv_k + (size_t)cl * kv_layer;
                    odd = (long)(kv_v - kv_k); pair = 16 * HD * 2; break;
                case ST_O: per = 8; sbase = lb + a.off_o + ((size_t)2 * r * KB_O + 8 * g) * 1024; odd = (long)KB_O * 1024; break;
                case ST_GU:
                    per = KBH; sbase = lb + a.off_gu + (size_t)t1 * KBH * 1024;
                    odd = (long)(t2 - t1) * KBH * 1024; half = true; break;
                case ST_D: per = 12; sbase = lb + a.off_d + ((size_t)2 * r * KB_D + 12 * g) * 1024; odd = (long)KB_D * 1024; break;
                default: break;
            }
            run_base();
        };
        auto issue_to = [&](int limit) {
            while (cg < limit) {
                if (ci >= cn) {
                    if (++cs == NSTAGE) { cs = 0; ++cl; }
                    if (cl >= L) break;
                    enter_stage();
                    continue;
                }
                // the rest of the current run, up to the limit (both even)
                const int n = min(per - rk, limit - cg);
                const bool act = !(half && (rj & 1)) || half_mine;
                const char* src = rbase + (rk + lid) * 1024 + lane * 16;
                for (int i = 0; i < n; i += 2) {
                    if (act)
                        __builtin_amdgcn_global_load_lds((const void*)src,
                                                         (__attribute__((address_space(3))) void*)(ring + (slot + lid) * 1024),
                                                         16, 0, NT);
                    src += 2048;
                    slot = slot + 2 == NSLOT ? 0 : slot + 2;
                }
                ci += n; cg += n; rk += n;
                if (rk >= per) { rk = 0; ++rj; run_base(); }
            }
        };
        int stage_begin = 0;       // global index of the first item of the barrier-phase stage
        issue_to(NSLOT);
        for (int l = 0; l < L; ++l) {
            for (int st = 0; st < NSTAGE; ++st) {
                const int n = sc.items(st), end = stage_begin + n;
                const int nb = n_barriers(st);
                for (int b = 0; b < nb; ++b) {
                    if (b == 0 && n > 0) {
                        // everything before this stage is released, so its remaining
                        // items fit; issue them, then wait for this loader's share
                        issue_to(end);
                        const int later = cg - end;
                        const int mine_later = (later + ((end & 1) == lid ? 1 : 0)) / 2;
                        wait_vm(mine_later < 40 ? mine_later : 40);
                        if (st == ST_D && lid == 0 && lane == 0 && l < TRACE_LAYERS)
                            ((unsigned long long*)(ws + wm.trace))[((((size_t)g * NRANK + r) * TRACE_LAYERS + l) * NSTAGE + ST_D) * 4 + 2] =
                                __builtin_amdgcn_s_memrealtime();
                    }
                    asm volatile("s_barrier" ::: "memory");
                    if (b == nb - 1) stage_begin = end;          // the stage's slots are released
                    // look ahead while the compute waves work, a bounded number
                    // of items per barrier interval: a long burst would keep
                    // this wave from the next barrier
                    issue_to(min(stage_begin + NSLOT, cg + LOOKAHEAD));
                }
            }
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        return;
    }

    // ------------------------------------------------------------------
    // Compute waves
    // ------------------------------------------------------------------
    int ring_base = 0;                   // global ring index of the current stage's first item
    const unsigned spin_limit = a.spin_limit;
    bool aborted = false;
    auto give_up = [&]() {
        atomicOr(a.status, PBD_STATUS_TIMEOUT);
        __hip_atomic_store(abort_w, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        aborted = true;
    };
    // wave 0, lanes 0..31: wait until all 32 ranks' flags of (flag kind, parity) hold tag
    // Polls keep three loads in flight per lane, so that a word is seen about
    // one round trip after it lands rather than up to two.
    auto wait_flags = [&](int fk, int p, unsigned tag) {
        if (wid != 0) return;
        const unsigned* f = (const unsigned*)(ws + wm.flags) + (((size_t)fk * 2 + p) * NGRP + g) * NRANK + (lane & (NRANK - 1));
        bool ok = lane >= NRANK;
        unsigned q[3];
#pragma unroll
        for (int k = 0; k < 3; ++k) q[k] = ld_sc1_u32(f);
        unsigned spins = 0;
        for (;;) {
            bool done = false;
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                ok = ok || q[k] == tag;
                if (__all(ok)) { done = true; break; }
                q[k] = ld_sc1_u32(f);
            }
            if (done) break;
            spins += 3;
            if (spins > spin_limit || ((spins & 63) < 3 && ld_sc1_u32(abort_w))) {
                if (lane == 0 && spins > spin_limit) give_up();
                break;
            }
        }
    };
    auto set_flag = [&](int fk, int p, unsigned tag) {
        // after this wave's (and, by the preceding barrier, every wave's) stores
        unsigned* f = (unsigned*)(ws + wm.flags) + (((size_t)fk * 2 + p) * NGRP + g) * NRANK + r;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __builtin_amdgcn_raw_buffer_store_b32(tag, rws, (unsigned)((char*)f - ws), 0, 0);
    };
    auto ring_frag = [&](int i) -> uint4 {
        return *(const uint4*)(ring + (size_t)((ring_base + i) % NSLOT) * 1024 + lane * 16);
    };
    // stage timestamps of every rank (profiling aid, 100 MHz clock): slot k
    // of stage st in layer l, written by lane 0 of the calling wave
    unsigned long long* trace = (unsigned long long*)(ws + wm.trace);
    auto stamp_at = [&](int l, int st, int k) {
        if (lane == 0 && l < TRACE_LAYERS)
            trace[((((size_t)g * NRANK + r) * TRACE_LAYERS + l) * NSTAGE + st) * 4 + k] = __builtin_amdgcn_s_memrealtime();
    };
    // after a stage's stores: every compute wave waits for its own, and the
    // last of them to arrive publishes the flag (and stamps slot 3 of stage st)
    auto publish = [&](int fk, int p, unsigned tag, int l, int st) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        unsigned old = 0;
        if (lane == 0) old = __hip_atomic_fetch_add(s_pub, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        old = __builtin_amdgcn_readfirstlane(old);
        if (old % NWC == NWC - 1) {
            if (lane == 0) set_flag(fk, p, tag);
            stamp_at(l, st, 3);
        }
    };
    f32x4* s_red = (f32x4*)scr;          // [tile][wave][mt][lane]
    // after barrier B: sum over waves w0..w0+nw-1 (in wave order) of tile tt's
    // accumulator quad holding rows n = 4 q .. 4 q + 3 of block row m
    auto red_quad = [&](int tt, int w0, int nw, int q, int m) -> f32x4 {
        const int mt = m / 16, ln = q * 16 + m % 16;
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int w = w0; w < w0 + nw; ++w) v += s_red[((tt * NWC + w) * 2 + mt) * WAVE + ln];
        return v;
    };
    const float* rope = (const float*)a.rope;
    const char* pk = (const char*)a.pk;
    const int MT = (M + 15) / 16;

    if (a.force_timeout && wid == 0) {
        // tests of the bounded wait: ctl[10] is never written
        unsigned spins = 0;
        while (ld_sc1_u32(ctl + 10) == 0u) {
            if (++spins > spin_limit) {
                if (lane == 0) give_up();
                break;
            }
        }
    }
    // residual slice from the assembled block (x [M][H], written by the previous kernel)
    for (int i = tid; i < MW * 32; i += NWC * WAVE) {
        const int m = i / 32, c = i % 32;
        xs[i] = m < M ? a.x0[(size_t)m * H + 32 * r + c] : 0.f;
    }

    auto stamp = [&](int l, int st, int k) {
        if (wid == 0) stamp_at(l, st, k);
    };
    // wave 0, lanes 0..7: wait until the last value producer group `lane`
    // writes into this rank's columns of layer pl's partial carries pl's tag
    // bit (its other values are checked one by one when read)
    auto wait_partials = [&](bool from_o, int pl) {
        if (wid != 0) return;
        const unsigned tb = ptag_bit(pl);
        const size_t base = (from_o ? wm.parto : wm.partd) + ((size_t)(pl & 1) * NGRP) * MW * H * 4;
        // system-scope loads: past this XCD's L2, which may hold the buffer's older contents
        const unsigned* pp = (const unsigned*)(ws + base + (((size_t)(lane % NGRP) * MW + (M - 1)) * H + 32 * r + 31) * 4);
        auto ldp = [&]() { return __hip_atomic_load(pp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) & 1u; };
        bool ok = lane >= NGRP;
        unsigned q[3];
#pragma unroll
        for (int k = 0; k < 3; ++k) q[k] = ldp();
        unsigned spins = 0;
        for (;;) {
            bool done = false;
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                ok = ok || q[k] == tb;
                if (__all(ok)) { done = true; break; }
                q[k] = ldp();
            }
            if (done) break;
            spins += 3;
            if (spins > spin_limit || ((spins & 63) < 3 && ld_sc1_u32(abort_w))) {
                if (lane == 0 && spins > spin_limit) give_up();
                break;
            }
        }
    };
    // R / R2 / final: residual update from the eight groups' partials (none at
    // layer 0's R), operand x * gain of the next RMSNorm and per-row sums of
    // squares.  Thread tid owns row tid / 16 (+ RR per round) and the column
    // pair 2 (tid % 16) of the rank's 32, so that every partial read is one
    // 16-byte load per group and a row's 16 column pairs sit in one DPP row.
    // `gv` is this thread's pair of gains (requested before the stage's wait).
    auto stage_reduce = [&](int l, bool from_o, float2 gv, size_t out_x, size_t out_sq, bool final_out) {
        const int p = l & 1;
        const bool poll = from_o || l > 0;
        // partials of layer l (O) or l - 1 (down) from every group
        const int pl = from_o ? l : l - 1;
        const unsigned tb = ptag_bit(pl);
        const unsigned base = (unsigned)((from_o ? wm.parto : wm.partd) + ((size_t)(pl & 1) * NGRP) * MW * H * 4);
        const int cp = tid % 16, c2 = 2 * cp;
        float2* xs2 = (float2*)xs;
#pragma unroll
        for (int e = 0; e < NRR; ++e) {
            if (e * RR >= M) break;
            const int m = tid / 16 + RR * e;
            const bool live = m < M;
            // all eight groups' pairs requested before any is used
            const unsigned voff = base + (unsigned)(((min(m, M - 1) * H) + 32 * r + c2) * 4);
            u32x2 q[NGRP];
            if (poll) {
#pragma unroll
                for (int x = 0; x < NGRP; ++x)
                    q[x] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rws, voff, x * MW * H * 4, SC01));
            }
            float2 xv = live ? xs2[m * 16 + cp] : float2{0.f, 0.f};
            if (poll && live) {
                float s0 = 0.f, s1 = 0.f;
#pragma unroll
                for (int x = 0; x < NGRP; ++x) {
                    u32x2 v = q[x];
                    // a value not yet written through: poll it alone (rare)
                    unsigned spins = 0;
                    while (((v.x & 1u) != tb) || ((v.y & 1u) != tb)) {
                        if (++spins > spin_limit || ((spins & 63) == 0 && ld_sc1_u32(abort_w))) {
                            if (spins > spin_limit) give_up();
                            v.x = 0u;
                            v.y = 0u;
                            break;
                        }
                        v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rws, voff, x * MW * H * 4, SC01));
                    }
                    // group order, the tag bit cleared (so that results do not
                    // depend on the pass's write count)
                    s0 += __uint_as_float(v.x & ~1u);
                    s1 += __uint_as_float(v.y & ~1u);
                }
                xv.x += s0;
                xv.y += s1;
                xs2[m * 16 + cp] = xv;
            }
            // operand and the row's sum of squares over the rank's 32 columns
            const float o0 = live ? xv.x * gv.x : 0.f, o1 = live ? xv.y * gv.y : 0.f;
            const float ss = row16_sum(xv.x * xv.x + xv.y * xv.y);
            if (final_out) {
                if (live) {
#pragma unroll
                    for (int k = 0; k < 2; ++k) {
                        const float ov = k == 0 ? o0 : o1;
                        const bf16 h = (bf16)ov;
                        const bf16 lo = (bf16)(ov - (float)h);
                        const size_t el = xfrag_elem<bf16>(m, 32 * r + c2 + k, a.lm_MT);
                        ((bf16*)a.lm_hi)[el] = h;
                        ((bf16*)a.lm_lo)[el] = lo;
                    }
                    if (cp == 0) a.lm_sq[(size_t)r * a.lm_sq_stride + m] = ss;
                }
            } else if (live) {
                const unsigned ooff = (unsigned)(out_x + ((size_t)p * NGRP + g) * MW * H * 4) + opnd_elem(m, 32 * r + c2);
                __builtin_amdgcn_raw_buffer_store_b32(f16_pair(o0, o1), rws, ooff, 0, 0);
                if (cp == 0)
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(ss), rws,
                        (unsigned)(out_sq + ((((size_t)p * NGRP + g) * MW + m) * NRANK + r) * 4), 0, 0);
            }
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };
    // this thread's pair of RMSNorm gains for stage_reduce
    auto gain_pair = [&](const void* gain) -> float2 {
        unsigned w;
        __builtin_memcpy(&w, (const bf16*)gain + 32 * r + 2 * (tid % 16), 4);
        return float2{(float)__builtin_bit_cast(bf16, (unsigned short)(w & 0xffff)),
                      (float)__builtin_bit_cast(bf16, (unsigned short)(w >> 16))};
    };

    // r_m of every row from the 32 ranks' partial sums of squares (wave 0, lanes < M)
    // in two phases, so that the operand loads issued in between overlap
    // them: lane (row m, half h) of wave 0 sums ranks 16 h .. 16 h + 15, which
    // lie next to each other ([parity][group][row][rank])
    auto rm_issue = [&](size_t sq_off, int p, u32x4 (&v)[NRANK / 8]) {
        if (wid == 0) {
            const int m = min(lane % MW, M - 1), h = lane / MW;
            const unsigned off = (unsigned)(sq_off + ((((size_t)p * NGRP + g) * MW + m) * NRANK + NRANK / 2 * h) * 4);
#pragma unroll
            for (int q = 0; q < NRANK / 8; ++q)
                v[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rws, off + 16 * q, 0, SC1));
        }
    };
    auto rm_finish = [&](const u32x4 (&v)[NRANK / 8]) {
        if (wid == 0) {
            float sm = 0.f;
#pragma unroll
            for (int q = 0; q < NRANK / 8; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e) sm += __uint_as_float(v[q][e]);
            sm += __shfl_xor(sm, MW, WAVE);
            if (lane < MW) s_rm[lane] = rsqrtf(sm / (float)H + a.eps);
        }
    };
    // The fp16 activation operands are stored fragment-major: fragment f of
    // m-tile mt is 1 KiB at byte (2 f + mt) * 1024, lane l's 16 bytes (row
    // l % 16, k-group l / 16) at l * 16, so one wavefront load reads 1 KiB of
    // contiguous memory.  Rows past the block are never written and stay zero.
    auto opnd_lane = [&](size_t base_off, int mt) -> unsigned {
        return (unsigned)(base_off + (size_t)mt * 1024 + (size_t)lane * 16);
    };
    // fp16 operand fragment fo bytes past the lane offset (fo: a wave-uniform constant)
    auto ld_frag = [&](unsigned voff, unsigned fo) -> uint4 {
        return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rws, voff, fo, SC1));
    };
    // the same for the second m-tile, where only the lanes of live rows issue
    // the load (for a 17-row block, one row in sixteen)
    auto ld_frag1 = [&](bool live, unsigned voff, unsigned fo) -> uint4 {
        uint4 x = uint4{0, 0, 0, 0};
        if (live) x = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rws, voff, fo, SC1));
        return x;
    };

    for (int l = 0; l < L; ++l) {
        // lane-derived offsets are recomputed in every layer instead of being
        // kept live (and spilled) across the whole loop
        asm volatile("" : "+v"(tid), "+v"(lane), "+v"(lrow), "+v"(lgrp));
        const int p = l & 1;
        const unsigned tag = (epoch << 8) | (unsigned)l;
        const size_t lay = (size_t)l * a.lay_stride;
        // The adapter's fragments do not depend on the activations: each
        // GEMM stage's LoRA A fragments and B block are requested one stage
        // ahead, so that they arrive (from HBM) while earlier stages wait.
        uint4 laQ[FPW], laO[3], laG[FPW], laU[FPW], laD[4];
        uint2 lbQ, lbO, lbG[2], lbD;

        // ---------------- R: residual from the down partials, attention-norm operand
        stamp(l, ST_R, 0);
        if (LORA) {
            const int src = sc.q_src();
            const uint32_t la_off = src == 0 ? a.off_la[0] : (src == 1 ? a.off_la[1] : a.off_la[2]);
            const uint4* la = (const uint4*)(pk + la_off + lay);
#pragma unroll
            for (int j = 0; j < FPW; ++j) laQ[j] = la[(size_t)min(wid + NWC * j, KBH - 1) * WAVE + lane];
            __builtin_memcpy(&lbQ, (const bf16*)(pk + a.off_lb_qkv + lay) + ((size_t)sc.q_tile() * WAVE + lane) * 4, 8);
        }
        {
            const float2 gv = gain_pair(pk + a.off_attn_norm + lay);
            if (l > 0) wait_partials(false, l - 1);
            bar();
            stamp(l, ST_R, 1);
            stage_reduce(l, false, gv, wm.xn, wm.sq, false);
        }
        publish(FL_R, p, tag, l, ST_R);

        // ---------------- Q: q/k/v tile
        stamp(l, ST_Q, 0);
        {
            wait_flags(FL_R, p, tag);
            bar();                                           // inputs ready, ring holds the tile
            stamp(l, ST_Q, 1);
            u32x4 rmv[NRANK / 8];
            rm_issue(wm.sq, p, rmv);
            const size_t xb = wm.xn + ((size_t)p * NGRP + g) * MW * H * 4;
            f32x4 acc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            f32x4 uacc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            // fragments f = wid + NWC j of the hidden size
            // fragments f = wid + NWC j (the last ones past the hidden size are
            // read from the next row and not used)
            uint4 xh[FPW][2];
            {
                const unsigned v0 = opnd_lane(xb, 0) + wid * 2048, v1 = opnd_lane(xb, 1) + wid * 2048;
                const bool live1 = 16 + lrow < M;
#pragma unroll
                for (int j = 0; j < FPW; ++j) {
                    xh[j][0] = ld_frag(v0, j * NWC * 2048);
                    xh[j][1] = ld_frag1(live1, v1, j * NWC * 2048);
                }
            }
            rm_finish(rmv);
#pragma unroll
            for (int j = 0; j < FPW; ++j) {
                if (wid + NWC * j >= KBH) continue;
                const f16x8 w = w_f16(ring_frag(wid + NWC * j));
                f16x8 ah;
                if (LORA) ah = w_f16(laQ[j]);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) {
                    if (mt >= MT) continue;
                    mma_h(acc[mt], w, xh[j][mt]);
                    if (LORA) mma_h(uacc[mt], ah, xh[j][mt]);
                }
            }
            if (LORA) {
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) if (mt < MT) mma_k4h(acc[mt], lbQ, uacc[mt] * a.scale);
            }
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) s_red[((0 * NWC + wid) * 2 + mt) * WAVE + lane] = acc[mt];
        }
        stamp(l, ST_Q, 2);
        bar();
        {
            // tile [16][M] -> qkv columns 16 r .. of the group's [M][512], four columns per thread
            const size_t qb = wm.qkv + ((size_t)p * NGRP + g) * MW * GQKV * 4;
            for (int i = tid; i < 4 * M; i += NWC * WAVE) {
                const int q = i % 4, m = i / 4;
                const f32x4 v = red_quad(0, 0, NWC, q, m) * s_rm[m];
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rws,
                    (unsigned)(qb + ((size_t)m * GQKV + 16 * r + 4 * q) * 4), 0, 0);
            }
            publish(FL_Q, p, tag, l, ST_Q);
        }
        ring_base += sc.items(ST_Q);

        // ---------------- A: attention split
        stamp(l, ST_A, 0);
        {
            bf16* q_l = (bf16*)scr;                                   // [QRMAX][LDQ]
            bf16* kb_l = (bf16*)(scr + QL_BYTES);                      // [32][LDQ]
            bf16* vb_l = (bf16*)(scr + QL_BYTES + KL_BYTES);           // [32][HD]
            float* pbuf = (float*)(scr + QL_BYTES + KL_BYTES + VL_BYTES);   // [4][16][PB]
            const bool blk = r == NRANK - 1;
            const size_t qb = wm.qkv + ((size_t)p * NGRP + g) * MW * GQKV * 4;
            typedef RowPrep<bf16, HD> RP;
            static_assert(RP::NP == 4, "row segments are 4 floats");
            auto ld4 = [&](size_t off) -> typename RP::fv {
                return __builtin_bit_cast(typename RP::fv, __builtin_amdgcn_raw_buffer_load_b128(rws, (unsigned)off, 0, SC1));
            };
            // Row jobs of 16 lanes each: the query rows q < QR (head q / M,
            // block row q % M), then (block split) the key rows and the value
            // rows of the block, or (verify, prefix splits) the key and value
            // rows r and r + 31 of the block that this rank appends to the
            // cache.  Lane group tg (of NG16) takes jobs tg + NG16 k, NJ at a
            // time; the position table and the norm gains are requested before
            // the wait, the q/k/v values after it.
            constexpr int NG16 = NWC * WAVE / 16, NJ = 3;
            const int tg = tid / 16;
            const int nkrow = blk ? ((M + 15) / 16) * 16 : 0;    // key rows incl. padding to the key block
            const int nkv = min(M, a.kv_rows);
            const int ncr = blk ? 0 : (r < nkv ? 1 : 0) + (r + NRANK - 1 < nkv ? 1 : 0);   // cache rows of this rank
            const int njob = QR + (blk ? 2 * M : 2 * ncr);
            Gains<bf16, HD> gq, gk;
            if (a.qk_norm) {
                gq.load(pk + a.off_q_norm + lay, lrow);
                gk.load(pk + a.off_k_norm + lay, lrow);
            }
            // job j: kind (0 query, 1 key, 2 value into LDS; 3 key, 4 value
            // into the cache), block row and source column
            auto job = [&](int j, int& kind, int& row, int& col) {
                if (j < QR) { kind = 0; row = j % M; col = (j / M) * HD; }
                else if (!blk) { const int c = j - QR; kind = 3 + (c & 1); row = r + (NRANK - 1) * (c >> 1); col = (2 + (c & 1)) * HD; }
                else if (j < QR + M) { kind = 1; row = j - QR; col = 2 * HD; }
                else { kind = 2; row = j - QR - M; col = 3 * HD; }
            };
            typename RP::fv2 cs[NJ];
#pragma unroll
            for (int k = 0; k < NJ; ++k) {
                int kind, row, col;
                job(min(tg + NG16 * k, njob - 1), kind, row, col);
                cs[k] = *(const typename RP::fv2*)((const float2*)rope + (size_t)(t + row) * RP::HALF + RP::NP * lrow);
            }
            wait_flags(FL_Q, p, tag);
            bar();
            stamp(l, ST_A, 1);
            float gql[RP::NP], gqh[RP::NP], gkl[RP::NP], gkh[RP::NP];
            gq.get(a.qk_norm, gql, gqh);
            gk.get(a.qk_norm, gkl, gkh);
            // the softmax scale (log2 e / sqrt(head_dim)) rides on the query
            // gains (the rotation is linear): the scores leave the MFMA scaled
#pragma unroll
            for (int pp = 0; pp < RP::NP; ++pp) {
                gql[pp] *= a.scale_log2;
                gqh[pp] *= a.scale_log2;
            }
            for (int j0 = 0; j0 < njob; j0 += NG16 * NJ) {
                typename RP::fv vlo[NJ], vhi[NJ];
#pragma unroll
                for (int k = 0; k < NJ; ++k) {
                    int kind, row, col;
                    job(min(j0 + tg + NG16 * k, njob - 1), kind, row, col);
                    const size_t rb = qb + ((size_t)row * GQKV + col + RP::NP * lrow) * 4;
                    vlo[k] = ld4(rb);
                    vhi[k] = ld4(rb + RP::HALF * 4);
                    if (j0 > 0)
                        cs[k] = *(const typename RP::fv2*)((const float2*)rope + (size_t)(t + row) * RP::HALF + RP::NP * lrow);
                }
#pragma unroll
                for (int k = 0; k < NJ; ++k) {
                    const int j = j0 + tg + NG16 * k;
                    if (j >= njob) continue;
                    int kind, row, col;
                    job(j, kind, row, col);
                    if (kind == 2) {
#pragma unroll
                        for (int pp = 0; pp < RP::NP; ++pp) {
                            vb_l[row * HD + RP::NP * lrow + pp] = (bf16)vlo[k][pp];
                            vb_l[row * HD + RP::HALF + RP::NP * lrow + pp] = (bf16)vhi[k][pp];
                        }
                    } else if (kind == 4) {
                        // value row for the cache: LDS row (row / 31) of the value
                        // buffer, which prefix splits do not use otherwise
                        const int cr = row / (NRANK - 1);
#pragma unroll
                        for (int pp = 0; pp < RP::NP; ++pp) {
                            vb_l[cr * HD + RP::NP * lrow + pp] = (bf16)vlo[k][pp];
                            vb_l[cr * HD + RP::HALF + RP::NP * lrow + pp] = (bf16)vhi[k][pp];
                        }
                    } else {
                        RP rp;
                        bf16 lo[RP::NP], hi[RP::NP];
                        rp.lo = vlo[k];
                        rp.hi = vhi[k];
                        rp.cs = cs[k];
                        float gl[RP::NP], gh[RP::NP];
#pragma unroll
                        for (int pp = 0; pp < RP::NP; ++pp) {
                            gl[pp] = kind == 0 ? gql[pp] : gkl[pp];
                            gh[pp] = kind == 0 ? gqh[pp] : gkh[pp];
                        }
                        // (a key row for the cache goes to LDS row (row / 31) of the
                        // key buffer, which prefix splits do not use otherwise)
                        rp.finish(kind == 0 ? q_l + j * LDQ : kb_l + (kind == 1 ? row : row / (NRANK - 1)) * LDQ, true, gl, gh,
                                  a.qk_norm, a.eps, lrow, lo, hi);
                    }
                }
            }
            // key and value rows past the block, up to the key block: zeros
            for (int i = tid; i < (nkrow - M) * HD; i += NWC * WAVE) {
                const int j = M + i / HD, d = i % HD;
                kb_l[j * LDQ + d] = (bf16)0.f;
                vb_l[j * HD + d] = (bf16)0.f;
            }
            bar();
            // key loop: wave w < 2 QT takes query tile w % QT and half w / QT of the blocks
            const int nb = blk ? (M + 15) / 16 : sc.kb_count();
            const int kb0 = sc.kb_begin();
            const int nparts = 2 * QT <= NWC ? 2 : 1;      // waves per query tile (key halves)
            const bool act = wid < nparts * QT;
            const int qt = wid % QT, half = wid / QT;
            const int hb = nparts == 2 ? (nb + 1) / 2 : nb;
            const int b_lo = half == 0 ? 0 : hb, b_hi = half == 0 ? hb : nb;
            f32x4 o_acc[HD / 16];
#pragma unroll
            for (int dt = 0; dt < HD / 16; ++dt) o_acc[dt] = f32x4{0, 0, 0, 0};
            float m_run = -1e30f, l_run = 0.f;
            const int qcol = qt * 16 + lrow;                  // query row of this lane's column
            const int jq = qcol < QR ? qcol % M : 0;
            if (act) {
                uint4 qf[HD / 32];
#pragma unroll
                for (int ds = 0; ds < HD / 32; ++ds) qf[ds] = *(const uint4*)(q_l + (qt * 16 + lrow) * LDQ + ds * 32 + lgrp * 8);
                bool first = true;
                for (int bi = b_lo; bi < b_hi; ++bi) {
                    uint4 kf[HD / 32];
                    uint2 vf[HD / 16];
                    if (blk) {
#pragma unroll
                        for (int ds = 0; ds < HD / 32; ++ds)
                            kf[ds] = *(const uint4*)(kb_l + (bi * 16 + lrow) * LDQ + ds * 32 + lgrp * 8);
#pragma unroll
                        for (int dt = 0; dt < HD / 16; ++dt) {
                            bf16 tmp[4];
#pragma unroll
                            for (int e = 0; e < 4; ++e) tmp[e] = vb_l[(bi * 16 + lgrp * 4 + e) * HD + dt * 16 + lrow];
                            __builtin_memcpy(&vf[dt], tmp, 8);
                        }
                    } else {
#pragma unroll
                        for (int ds = 0; ds < HD / 32; ++ds) kf[ds] = ring_frag(bi * 8 + ds);
#pragma unroll
                        for (int dt = 0; dt < HD / 16; ++dt)
                            vf[dt] = *(const uint2*)(ring + (size_t)((ring_base + bi * 8 + 4 + dt / 2) % NSLOT) * 1024 +
                                                     (dt % 2) * 512 + lane * 8);
                    }
                    f32x4 s = f32x4{0, 0, 0, 0};
#pragma unroll
                    for (int ds = 0; ds < HD / 32; ++ds) mma_frag<bf16>(s, kf[ds], qf[ds]);
                    float sv[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int kk = bi * 16 + lgrp * 4 + e;
                        bool ok;
                        if (blk) ok = kk < M && (kk <= jq || jq >= a.full_from);
                        else ok = (kb0 * 16 + kk) < t;
                        ok = ok && qcol < QR;
                        sv[e] = ok ? s[e] : -INFINITY;
                    }
                    float mloc = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
                    mloc = xrow_max(mloc);
                    const float m_new = fmaxf(m_run, mloc);
                    if (!first) {
                        const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
                        l_run *= corr;
#pragma unroll
                        for (int dt = 0; dt < HD / 16; ++dt) o_acc[dt] *= corr;
                    }
                    first = false;
                    m_run = m_new;
                    f32x4 pr;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        pr[e] = __builtin_amdgcn_exp2f(sv[e] - m_run);
                        l_run += pr[e];
                    }
#pragma unroll
                    for (int dt = 0; dt < HD / 16; ++dt) mma_k4(o_acc[dt], vf[dt], pr);
                }
                l_run = xrow_sum(l_run);
                if (half == 1) {
                    float* pb = pbuf + (size_t)(qt * 16 + lrow) * PB;
                    if (lgrp == 0) { pb[HD] = m_run; pb[HD + 1] = l_run; }
#pragma unroll
                    for (int dt = 0; dt < HD / 16; ++dt) *(f32x4*)(pb + dt * 16 + lgrp * 4) = o_acc[dt];
                }
            }
            bar();
            if (act && half == 0) {
                // merge with the other half (if it had blocks) in place of the pair buffer
                float* pb = pbuf + (size_t)(qt * 16 + lrow) * PB;
                float m1 = -1e30f, l1 = 0.f;
                const bool other = b_hi < nb;
                if (other) { m1 = pb[HD]; l1 = pb[HD + 1]; }
                const float mx = fmaxf(m_run, m1);
                const float f0 = __builtin_amdgcn_exp2f(m_run - mx), f1 = other ? __builtin_amdgcn_exp2f(m1 - mx) : 0.f;
#pragma unroll
                for (int dt = 0; dt < HD / 16; ++dt) {
                    f32x4 o1 = other ? *(const f32x4*)(pb + dt * 16 + lgrp * 4) : f32x4{0, 0, 0, 0};
                    o_acc[dt] = o_acc[dt] * f0 + o1 * f1;
                }
                const float ltot = l_run * f0 + l1 * f1;
                // a column with no visible key keeps max -inf and sum 0
                const bool any = ltot > 0.f;
#pragma unroll
                for (int dt = 0; dt < HD / 16; ++dt) *(f32x4*)(pb + dt * 16 + lgrp * 4) = o_acc[dt];
                if (lgrp == 0) { pb[HD] = any ? mx : -INFINITY; pb[HD + 1] = any ? ltot : 0.f; }
            }
            bar();
            {
                // partial of split r for every query row: (m, l, o[128])
                const size_t ab0 = wm.apart + ((((size_t)p * NGRP + g) * NRANK + r) * QRMAX) * APW * 4;
                const bool has = nb > 0;
                for (int i = tid; i < QR * (HD / 4 + 1); i += NWC * WAVE) {
                    const int q = i / (HD / 4 + 1), c4 = i % (HD / 4 + 1);
                    const float* pb = pbuf + (size_t)q * PB;
                    f32x4 v;
                    if (c4 < HD / 4) v = has ? *(const f32x4*)(pb + c4 * 4) : f32x4{0, 0, 0, 0};
                    else v = f32x4{has ? pb[HD] : -INFINITY, has ? pb[HD + 1] : 0.f, 0.f, 0.f};
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rws,
                        (unsigned)(ab0 + ((size_t)q * APW + (c4 < HD / 4 ? 4 + c4 * 4 : 0)) * 4), 0, 0);
                }
                publish(FL_A, p, tag, l, ST_A);
            }
        }
        ring_base += sc.items(ST_A);

        // ---------------- M: merge the 32 split partials of query rows r, r + 32
        stamp(l, ST_M, 0);
        if (LORA) {
            const int tt = wid / 3, f0 = wid % 3;
            const uint4* la = (const uint4*)(pk + a.off_la[3] + lay);
#pragma unroll
            for (int j = 0; j < 3; ++j) laO[j] = la[(size_t)(8 * g + min(f0 + 3 * j, 7)) * WAVE + lane];
            __builtin_memcpy(&lbO, (const bf16*)(pk + a.off_lb_o + lay) + ((size_t)(2 * r + tt) * WAVE + lane) * 4, 8);
        }
        wait_flags(FL_A, p, tag);
        bar();
        stamp(l, ST_M, 1);
        if (wid < 2) {
            const int q = r + 32 * wid;
            if (q < QR) {
                const unsigned ab = (unsigned)(wm.apart + (((size_t)p * NGRP + g) * NRANK) * QRMAX * APW * 4);
                // every split's (m, l) (lane s < 32 holds split s's) and this
                // lane's two dims of every split's o, all requested at once
                uint2 ml = uint2{__float_as_uint(-INFINITY), 0u};
                if (lane < NRANK)
                    ml = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rws,
                        ab + (unsigned)(((size_t)lane * QRMAX + q) * APW * 4), 0, SC1));
                uint2 ov[NRANK];
                const unsigned ob0 = ab + (unsigned)(((size_t)q * APW + 4 + 2 * lane) * 4);
#pragma unroll
                for (int k = 0; k < NRANK; ++k)
                    ov[k] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rws, ob0, k * QRMAX * APW * 4, SC1));
                const float mls = __uint_as_float(ml.x);
                const float mx = wave_max(mls);
                const float wl = (mls > -INFINITY) ? __builtin_amdgcn_exp2f(mls - mx) : 0.f;
                const float wll = wl * __uint_as_float(ml.y);
                // merged in fixed split order, the weights read from their lanes
                float o0 = 0.f, o1 = 0.f, Ls = 0.f;
#pragma unroll
                for (int k = 0; k < NRANK; ++k) {
                    const float w = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__float_as_uint(wl), k));
                    o0 += w * __uint_as_float(ov[k].x);
                    o1 += w * __uint_as_float(ov[k].y);
                    Ls += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__float_as_uint(wll), k));
                }
                const float inv = Ls > 0.f ? 1.f / Ls : 0.f;
                const int hl = q / M, j = q % M;
                const size_t ob = wm.oop + ((size_t)p * NGRP + g) * MW * GO * 4;
                const unsigned ooff = (unsigned)ob + opnd_elem(j, hl * HD + 2 * lane);
                __builtin_amdgcn_raw_buffer_store_b32(f16_pair(o0 * inv, o1 * inv), rws, ooff, 0, 0);
            }
        }
        publish(FL_M, p, tag, l, ST_M);
        {
            // verify: this rank's rows r and r + 31 of the block K/V (kept in
            // LDS since the attention stage) appended to the cache at t + row,
            // after the flag, so that the stores stay off the stage chain
            const int nkv = min(M, a.kv_rows);
            const int ncr = r == NRANK - 1 ? 0 : (r < nkv ? 1 : 0) + (r + NRANK - 1 < nkv ? 1 : 0);
            const bf16* kb_l = (const bf16*)(scr + QL_BYTES);
            const bf16* vb_l = (const bf16*)(scr + QL_BYTES + KL_BYTES);
            const size_t head = (((size_t)l * a.Bmax) * NKV + g) * (size_t)a.nblk * 16 * HD;
            for (int i = tid; i < ncr * HD; i += NWC * WAVE) {
                const int cr = i / HD, dd = i % HD, pos = t + r + (NRANK - 1) * cr;
                bf16* kblk = (bf16*)a.kcache + head + (size_t)(pos / 16) * 16 * HD;
                bf16* vblk = (bf16*)a.vcache + head + (size_t)(pos / 16) * 16 * HD;
                kblk[kblock_elem<bf16>(pos % 16, dd)] = kb_l[cr * LDQ + dd];
                vblk[vblock_elem(pos % 16, dd)] = vb_l[cr * HD + dd];
            }
        }

        // ---------------- O: O-projection partial over the group's heads
        stamp(l, ST_O, 0);
        {
            // tile tt = wid / 3; fragments f = wid % 3 + 3 j of the group's 8
            const int tt = wid / 3, f0 = wid % 3;
            wait_flags(FL_M, p, tag);
            bar();
            stamp(l, ST_O, 1);
            const size_t ob = wm.oop + ((size_t)p * NGRP + g) * MW * GO * 4;
            f32x4 acc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            f32x4 uacc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            // fragments f0 + 3 j of the group's 8 (f = 8 is read from the next row, unused)
            uint4 xh[3][2];
            {
                const unsigned v0 = opnd_lane(ob, 0) + f0 * 2048, v1 = opnd_lane(ob, 1) + f0 * 2048;
                const bool live1 = 16 + lrow < M;
#pragma unroll
                for (int j = 0; j < 3; ++j) {
                    xh[j][0] = ld_frag(v0, j * 3 * 2048);
                    xh[j][1] = ld_frag1(live1, v1, j * 3 * 2048);
                }
            }
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                if (f0 + 3 * j >= 8) continue;
                const f16x8 w = w_f16(ring_frag(tt * 8 + f0 + 3 * j));
                f16x8 ah;
                if (LORA) ah = w_f16(laO[j]);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) {
                    if (mt >= MT) continue;
                    mma_h(acc[mt], w, xh[j][mt]);
                    if (LORA) mma_h(uacc[mt], ah, xh[j][mt]);
                }
            }
            if (LORA) {
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) if (mt < MT) mma_k4h(acc[mt], lbO, uacc[mt] * a.scale);
            }
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) s_red[((tt * NWC + wid) * 2 + mt) * WAVE + lane] = acc[mt];
        }
        stamp(l, ST_O, 2);
        bar();
        {
            // partial [M][32 columns], tagged, written through to memory
            const size_t pb = wm.parto + (((size_t)p * NGRP + g) * MW) * H * 4;
            const unsigned tb = ptag_bit(l);
            for (int i = tid; i < 8 * M; i += NWC * WAVE) {
                // columns 16 tt + 4 q .. + 3 of the rank's 32, each value's lowest bit the tag
                const int m = i / 8, tt = (i % 8) / 4, q = i % 4;
                const f32x4 v = red_quad(tt, tt * 3, 3, q, m);
                const unsigned off = (unsigned)(pb + ((size_t)m * H + 32 * r + 16 * tt + 4 * q) * 4);
                __builtin_amdgcn_raw_buffer_store_b128(u32x4{(__float_as_uint(v[0]) & ~1u) | tb, (__float_as_uint(v[1]) & ~1u) | tb,
                                                             (__float_as_uint(v[2]) & ~1u) | tb, (__float_as_uint(v[3]) & ~1u) | tb},
                                                       rws, off, 0, SC1);
            }
        }
        ring_base += sc.items(ST_O);

        // ---------------- R2: residual from the O partials, MLP-norm operand
        stamp(l, ST_R2, 0);
        if (LORA) {
            const uint4* lag = (const uint4*)(pk + a.off_la[4] + lay);
            const uint4* lau = (const uint4*)(pk + a.off_la[5] + lay);
#pragma unroll
            for (int j = 0; j < FPW; ++j) {
                const int f = min(wid + NWC * j, KBH - 1);
                laG[j] = lag[(size_t)f * WAVE + lane];
                laU[j] = lau[(size_t)f * WAVE + lane];
            }
#pragma unroll
            for (int tt = 0; tt < 2; ++tt)
                __builtin_memcpy(&lbG[tt], (const bf16*)(pk + a.off_lb_gu + lay) +
                                               ((size_t)(tt == 0 ? sc.gu_t1() : sc.gu_t2()) * WAVE + lane) * 4, 8);
        }
        {
            const float2 gv = gain_pair(pk + a.off_mlp_norm + lay);
            wait_partials(true, l);
            bar();
            stamp(l, ST_R2, 1);
            stage_reduce(l, true, gv, wm.xm, wm.sqm, false);
        }
        publish(FL_R2, p, tag, l, ST_R2);

        // ---------------- GU: gate/up tiles + SwiGLU
        stamp(l, ST_GU, 0);
        {
            // the down stage's adapter fragments, one stage ahead
            if (LORA) {
                const int tt = wid / 3, f0 = wid % 3;
                const uint4* la = (const uint4*)(pk + a.off_la[6] + lay);
#pragma unroll
                for (int j = 0; j < 4; ++j) laD[j] = la[(size_t)(12 * g + f0 + 3 * j) * WAVE + lane];
                __builtin_memcpy(&lbD, (const bf16*)(pk + a.off_lb_d + lay) + ((size_t)(2 * r + tt) * WAVE + lane) * 4, 8);
            }
            wait_flags(FL_R2, p, tag);
            bar();
            stamp(l, ST_GU, 1);
            u32x4 rmv[NRANK / 8];
            rm_issue(wm.sqm, p, rmv);
            const size_t xb = wm.xm + ((size_t)p * NGRP + g) * MW * H * 4;
            f32x4 acc[2][2] = {{f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}}, {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}}};
            f32x4 ug[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}}, uu[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            const bool mine2 = ((lrow / 4) & 1) == (r & 1);
            // fragments f = wid + NWC j (the last ones past the hidden size are
            // read from the next row and not used)
            uint4 xh[FPW][2];
            {
                const unsigned v0 = opnd_lane(xb, 0) + wid * 2048, v1 = opnd_lane(xb, 1) + wid * 2048;
                const bool live1 = 16 + lrow < M;
#pragma unroll
                for (int j = 0; j < FPW; ++j) {
                    xh[j][0] = ld_frag(v0, j * NWC * 2048);
                    xh[j][1] = ld_frag1(live1, v1, j * NWC * 2048);
                }
            }
            rm_finish(rmv);
#pragma unroll
            for (int j = 0; j < FPW; ++j) {
                const int f = wid + NWC * j;
                if (f >= KBH) continue;
                const f16x8 w1 = w_f16(ring_frag(f));
                const f16x8 w2 = w_f16(mine2 ? ring_frag(KBH + f) : uint4{0, 0, 0, 0});
                f16x8 gh, uh;
                if (LORA) {
                    gh = w_f16(laG[j]);
                    uh = w_f16(laU[j]);
                }
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) {
                    if (mt >= MT) continue;
                    mma_h(acc[0][mt], w1, xh[j][mt]);
                    mma_h(acc[1][mt], w2, xh[j][mt]);
                    if (LORA) {
                        mma_h(ug[mt], gh, xh[j][mt]);
                        mma_h(uu[mt], uh, xh[j][mt]);
                    }
                }
            }
            if (LORA) {
#pragma unroll
                for (int tt = 0; tt < 2; ++tt) {
                    const uint2 bv = lbG[tt];
                    // rows 0-7 take the gate shrink, rows 8-15 the up shrink
                    const uint2 bg = lrow < 8 ? bv : uint2{0, 0};
                    const uint2 bu = lrow < 8 ? uint2{0, 0} : bv;
#pragma unroll
                    for (int mt = 0; mt < 2; ++mt) {
                        if (mt >= MT) continue;
                        mma_k4h(acc[tt][mt], bg, ug[mt] * a.scale);
                        mma_k4h(acc[tt][mt], bu, uu[mt] * a.scale);
                    }
                }
            }
#pragma unroll
            for (int tt = 0; tt < 2; ++tt)
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) s_red[((tt * NWC + wid) * 2 + mt) * WAVE + lane] = acc[tt][mt];
        }
        stamp(l, ST_GU, 2);
        bar();
        {
            // h for the rank's 12 FFN columns: 8 from the full tile, 4 from the half tile
            const size_t hb = wm.hop + ((size_t)p * NGRP + g) * MW * GF * 4;
            // (four adjacent columns per thread: gate rows 4 q .. 4 q + 3 of the
            // tile, up rows 8 + 4 q ..)
            for (int i = tid; i < 3 * M; i += NWC * WAVE) {
                const int m = i / 3, jq = i % 3;
                const int tt = jq < 2 ? 0 : 1, q = jq < 2 ? jq : (r & 1);
                const int col = jq < 2 ? 8 * r + 4 * jq : 256 + 4 * r;
                const float rm = s_rm[m];
                const f32x4 gq = red_quad(tt, 0, NWC, q, m), uq = red_quad(tt, 0, NWC, q + 2, m);
                float hv[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float gt = gq[e] * rm;
                    const float up = uq[e] * rm;
                    hv[e] = gt / (1.f + __expf(-gt)) * up;
                }
                const unsigned ooff = (unsigned)hb + opnd_elem(m, col);
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{f16_pair(hv[0], hv[1]), f16_pair(hv[2], hv[3])}, rws, ooff, 0, 0);
            }
            publish(FL_GU, p, tag, l, ST_GU);
        }
        ring_base += sc.items(ST_GU);

        // ---------------- D: down-projection partial over the group's FFN slice
        stamp(l, ST_D, 0);
        {
            // tile tt = wid / 3; fragments f = wid % 3 + 3 j of the group's 12
            const int tt = wid / 3, f0 = wid % 3;
            wait_flags(FL_GU, p, tag);
            bar();
            stamp(l, ST_D, 1);
            const size_t hb = wm.hop + ((size_t)p * NGRP + g) * MW * GF * 4;
            f32x4 acc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            f32x4 uacc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
            uint4 xh[4][2];
            {
                const unsigned v0 = opnd_lane(hb, 0) + f0 * 2048, v1 = opnd_lane(hb, 1) + f0 * 2048;
                const bool live1 = 16 + lrow < M;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    xh[j][0] = ld_frag(v0, j * 3 * 2048);
                    xh[j][1] = ld_frag1(live1, v1, j * 3 * 2048);
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f16x8 w = w_f16(ring_frag(tt * 12 + f0 + 3 * j));
                f16x8 ah;
                if (LORA) ah = w_f16(laD[j]);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) {
                    if (mt >= MT) continue;
                    mma_h(acc[mt], w, xh[j][mt]);
                    if (LORA) mma_h(uacc[mt], ah, xh[j][mt]);
                }
            }
            if (LORA) {
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) if (mt < MT) mma_k4h(acc[mt], lbD, uacc[mt] * a.scale);
            }
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) s_red[((tt * NWC + wid) * 2 + mt) * WAVE + lane] = acc[mt];
        }
        bar();
        {
            const size_t pb = wm.partd + (((size_t)p * NGRP + g) * MW) * H * 4;
            const unsigned tb = ptag_bit(l);
            for (int i = tid; i < 8 * M; i += NWC * WAVE) {
                // columns 16 tt + 4 q .. + 3 of the rank's 32, each value's lowest bit the tag
                const int m = i / 8, tt = (i % 8) / 4, q = i % 4;
                const f32x4 v = red_quad(tt, tt * 3, 3, q, m);
                const unsigned off = (unsigned)(pb + ((size_t)m * H + 32 * r + 16 * tt + 4 * q) * 4);
                __builtin_amdgcn_raw_buffer_store_b128(u32x4{(__float_as_uint(v[0]) & ~1u) | tb, (__float_as_uint(v[1]) & ~1u) | tb,
                                                             (__float_as_uint(v[2]) & ~1u) | tb, (__float_as_uint(v[3]) & ~1u) | tb},
                                                       rws, off, 0, SC1);
            }
        }
        ring_base += sc.items(ST_D);
    }
    // final RMSNorm operand of the LM head (group 0 writes it)
    stamp(L, 0, 0);
    if (g == 0) stage_reduce(L, false, gain_pair(a.final_norm), 0, 0, true);
    stamp(L, 0, 1);
}

}  // namespace fz

size_t fused_ws_bytes() { return fz::ws_map().total; }
size_t fused_ctl_offset() { return fz::ws_map().ctl; }
size_t fused_trace_offset() { return fz::ws_map().trace; }
int fused_trace_entries() { return fz::NGRP * fz::NRANK * fz::TRACE_LAYERS * fz::NSTAGE * 4; }
size_t fused_lds_bytes() { return fz::LDS_BYTES; }
int fused_threads() { return fz::NTHR; }

hipError_t fused_occupancy(int* blocks_per_cu) {
    hipError_t e = hipFuncSetAttribute((const void*)fz::k_fused<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)fz::LDS_BYTES);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute((const void*)fz::k_fused<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)fz::LDS_BYTES);
    if (e != hipSuccess) return e;
    int a = 0, b = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, fz::k_fused<false>, fz::NTHR, fz::LDS_BYTES);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, fz::k_fused<true>, fz::NTHR, fz::LDS_BYTES);
    if (e != hipSuccess) return e;
    *blocks_per_cu = a < b ? a : b;
    return hipSuccess;
}

hipError_t launch_fused(const FusedArgs& a, bool lora, hipStream_t st) {
    if (a.M < 1 || a.M > FUSED_MAX_ROWS || a.L < 1 || a.L > 255) return hipErrorInvalidValue;
    static bool attr_set[2] = {false, false};
    auto kern = lora ? (const void*)fz::k_fused<true> : (const void*)fz::k_fused<false>;
    if (!attr_set[lora ? 1 : 0]) {
        hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)fz::LDS_BYTES);
        if (e != hipSuccess) return e;
        attr_set[lora ? 1 : 0] = true;
    }
    hipEvent_t e0 = nullptr, e1 = nullptr;
    get_launch_events(&e0, &e1);
    if (e0) {
        if (lora) hipExtLaunchKernelGGL((fz::k_fused<true>), dim3(256), dim3(fz::NTHR), fz::LDS_BYTES, st, e0, e1, 0, a);
        else hipExtLaunchKernelGGL((fz::k_fused<false>), dim3(256), dim3(fz::NTHR), fz::LDS_BYTES, st, e0, e1, 0, a);
    } else {
        if (lora) hipLaunchKernelGGL((fz::k_fused<true>), dim3(256), dim3(fz::NTHR), fz::LDS_BYTES, st, a);
        else hipLaunchKernelGGL((fz::k_fused<false>), dim3(256), dim3(fz::NTHR), fz::LDS_BYTES, st, a);
    }
    return hipGetLastError();
}

}  // namespace pbd
