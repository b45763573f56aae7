// Streaming append of one token per (sequence, kv head) into the sink or the residual
// (Fig. 4 pseudo-decode; App. D three-region cache).  One workgroup per sequence: every
// thread reads the sequence's length before the copy and thread 0 publishes length + 1 after
// a barrier, so all kv heads of a sequence use the same slot.
#include "common.hpp"

namespace kvarn {
namespace {

struct AppendArgs {
    kvarn_cache c;
    int n_sink;
    const void* k_new;
    const void* v_new;
    int bf16;
};

__global__ __launch_bounds__(256) void k_append(AppendArgs a) {
    const int b = blockIdx.x;
    const int len = a.c.seq_len[b];
    const bool sink = len < a.n_sink;
    int slot = len;
    if (len < 0) {  // corrupted length: refuse rather than index with it
        if (threadIdx.x == 0 && a.c.err_word)
            __hip_atomic_fetch_or(a.c.err_word, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    if (!sink) {
        const int r = (len - a.n_sink) % kG, nb = (len - a.n_sink) / kG;
        if (r == kG - 1 && nb >= a.c.max_blocks) {  // the flush would need a missing body tile
            if (threadIdx.x == 0 && a.c.err_word)
                __hip_atomic_fetch_or(a.c.err_word, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
        slot = r;
    }
    // 2 * n_kv rows of 128 elements; each thread moves 4 elements (8 bytes of bf16)
    const int n_chunks = a.c.n_kv * 2 * (kD / 4);
    for (int idx = threadIdx.x; idx < n_chunks; idx += blockDim.x) {
        const int row = idx / (kD / 4), c4 = (idx % (kD / 4)) * 4;
        const int kvh = row >> 1, is_v = row & 1;
        const size_t stream = (size_t)b * a.c.n_kv + kvh;
        const size_t src = stream * kD + c4;
        uint16_t h[4];
        if (a.bf16) {
            const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(is_v ? a.v_new : a.k_new) + src);
            h[0] = (uint16_t)v.x; h[1] = (uint16_t)(v.x >> 16); h[2] = (uint16_t)v.y; h[3] = (uint16_t)(v.y >> 16);
        } else {
            const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(is_v ? a.v_new : a.k_new) + src);
            h[0] = f32_to_bf16(v.x); h[1] = f32_to_bf16(v.y); h[2] = f32_to_bf16(v.z); h[3] = f32_to_bf16(v.w);
        }
        uint16_t* dst;
        if (sink)
            dst = static_cast<uint16_t*>(is_v ? a.c.v_sink : a.c.k_sink) + (stream * a.n_sink + slot) * kD + c4;
        else
            dst = static_cast<uint16_t*>(is_v ? a.c.v_resid : a.c.k_resid) + (stream * kG + slot) * kD + c4;
        *reinterpret_cast<uint2*>(dst) = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16),
                                                    (uint32_t)h[2] | ((uint32_t)h[3] << 16));
    }
    __syncthreads();
    if (threadIdx.x == 0) a.c.seq_len[b] = len + 1;
}

}  // namespace

hipError_t launch_append(const kvarn_cache& c, int n_sink, const void* k_new, const void* v_new, bool bf16,
                         hipStream_t stream) {
    AppendArgs a{c, n_sink, k_new, v_new, bf16 ? 1 : 0};
    hipLaunchKernelGGL(k_append, dim3((unsigned)c.batch), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace kvarn
