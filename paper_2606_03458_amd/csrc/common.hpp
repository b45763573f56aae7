// Shared device/host definitions of libkvarn (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvarn.h"

namespace kvarn {

constexpr int kD = 128;  // head_dim (channels per token)
constexpr int kG = 128;  // tokens per quantization group / body tile
constexpr int64_t kMaxStreams = int64_t(1) << 26;  // (sequence, kv head) pairs a cache may hold

// 1/sqrt(128), rounded to fp32.
constexpr float kInvSqrt128 = 0.08838834764831845f;
constexpr float kLog2e = 1.4426950408889634f;

// aux bytes per tile: three fp32 vectors, or the compact binary16 b + E4M3 a + E4M3 s2
__host__ __device__ inline size_t aux_bytes(int compact) { return compact ? 512 : 3 * 128 * sizeof(float); }
__host__ __device__ inline size_t code_bytes(int bits) { return (size_t)bits * 2048; }
__host__ __device__ inline size_t tile_bytes(int bits, int compact) { return code_bytes(bits) + aux_bytes(compact); }

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Quantizer constants, as passed to kernels.
struct QParams {
    int bits;
    int iters;
    float var_min, var_max, log_lo, log_hi;
    int compact;  // aux format: 0 fp32, 1 compact
    int rotate;   // 1: Hadamard rotation along head_dim before VarN; 0: none (ablations)
};

// Kernel launchers (defined in the .hip files; called by the host API).
hipError_t launch_quantize_tiles(const QParams& qp, int kind, const void* x, bool x_bf16, int64_t n_outer,
                                 int64_t n_inner, int64_t x_outer, int64_t x_inner, int64_t x_token, void* out,
                                 int64_t out_outer, int64_t out_inner, int32_t* best_iter, hipStream_t stream);

// all_due: the caller knows every sequence completes a group with this token (lock-step
// decode): one workgroup per tile.  Otherwise a resident-size grid checks the tiles.
hipError_t launch_flush(const QParams& qp, const kvarn_cache& c, int n_sink, bool all_due, hipStream_t stream);

hipError_t launch_prefill(const QParams& qp, const kvarn_cache& c, int n_sink, const void* k, const void* v,
                          bool x_bf16, const int32_t* cu_seqlens, int max_len, hipStream_t stream);

hipError_t launch_append(const kvarn_cache& c, int n_sink, const void* k_new, const void* v_new, bool bf16,
                         hipStream_t stream);

struct DecodePlan {
    int n_chunk, g_chunk;  // query heads of a group taken in n_chunk chunks of up to g_chunk (<= 8)
    int n_split;           // splits per (sequence, kv head)
    int n_res;             // splits (the last of n_split) that hold only sink + residual chunks
    int group;             // > 1: the n_split splits of a stream are the waves of one workgroup
    int blocks_per_split;  // body tiles per body split
    int max_blocks_used;   // upper bound of body tiles over the batch
};

DecodePlan plan_decode(int batch, int n_kv, int n_q, int bits, int max_len, int n_sink, int max_blocks);
size_t decode_workspace_bytes(int batch, int n_q, const DecodePlan& plan);

// A lock-step decode step's token, appended by the decode launch itself (bf16 rows [batch][n_kv][128],
// 16-byte aligned; len_before >= n_sink and the token does not fill the residual).
struct StepAppend {
    int len_before;
    const void* k_new;
    const void* v_new;
};
hipError_t launch_decode(const kvarn_cache& c, int bits, int compact, int rotate, int n_sink, int n_q, const void* q,
                         bool q_bf16, void* out, bool out_bf16, float sm_scale, const DecodePlan& plan, float* ws,
                         hipStream_t stream, const StepAppend* step = nullptr);

}  // namespace kvarn
