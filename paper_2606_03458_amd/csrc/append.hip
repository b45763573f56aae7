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
    // A corrupted length, or a flush that would need a missing body tile: refuse (flag, no
    // store).  The token's values are loaded before this is known (their addresses do not depend
    // on the length), so the length and the values arrive in one memory round trip.
    const bool sink = len < a.n_sink;
    const int r = (len - a.n_sink) % kG, nb = (len - a.n_sink) / kG;
    const bool bad = len < 0 || (!sink && r == kG - 1 && nb >= a.c.max_blocks);
    const int slot = sink ? len : r;
    // 2 * n_kv rows of 128 elements; each thread moves 4 elements (8 bytes of bf16), U chunks at
    // a time with all their loads in flight before the first store
    constexpr int U = 4;
    const int n_chunks = a.c.n_kv * 2 * (kD / 4);
    for (int base = 0; base < n_chunks; base += U * blockDim.x) {
        uint32_t w[U][2];
        size_t src[U];
        bool vrow[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int idx = min(base + u * (int)blockDim.x + (int)threadIdx.x, n_chunks - 1);
            const int row = idx / (kD / 4), c4 = (idx % (kD / 4)) * 4;
            src[u] = ((size_t)b * a.c.n_kv + (row >> 1)) * kD + c4;
            vrow[u] = row & 1;
        }
        if (a.bf16) {  // one branch on the dtype, so every load of the batch is in flight at once
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(vrow[u] ? a.v_new : a.k_new) + src[u]);
                w[u][0] = v.x;
                w[u][1] = v.y;
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(vrow[u] ? a.v_new : a.k_new) + src[u]);
                w[u][0] = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
                w[u][1] = (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
            }
        }
        if (bad) continue;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int idx = base + u * (int)blockDim.x + (int)threadIdx.x;
            if (idx >= n_chunks) break;
            const int row = idx / (kD / 4), c4 = (idx % (kD / 4)) * 4;
            const size_t stream = (size_t)b * a.c.n_kv + (row >> 1);
            const bool is_v = row & 1;
            uint16_t* dst;
            if (sink)
                dst = static_cast<uint16_t*>(is_v ? a.c.v_sink : a.c.k_sink) + (stream * a.n_sink + slot) * kD + c4;
            else
                dst = static_cast<uint16_t*>(is_v ? a.c.v_resid : a.c.k_resid) + (stream * kG + slot) * kD + c4;
            *reinterpret_cast<uint2*>(dst) = make_uint2(w[u][0], w[u][1]);
        }
    }
    if (bad) {
        if (threadIdx.x == 0 && a.c.err_word)
            __hip_atomic_fetch_or(a.c.err_word, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
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
