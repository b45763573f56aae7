// KVarN decode attention for gfx950 (App. D three-region cache, App. I fused second scale,
// App. A rotation layout).
//
// Body (quantized) tokens are attended in the rotated domain: with q_rot = H q and the packed
// tile's aux, a key's logit is
//     s2K[t] * (sum_c q_rot[c] a_K[c] code[t][c] + sum_c q_rot[c] b_K[c])
// and a value tile adds  s2V[c] * (sum_t p[t] a_V[t] code[t][c] + sum_t p[t] b_V[t])  to the
// rotated output, so each body tile costs one pass over its codes with both scales fused.
// Sink and residual tokens (bf16, unrotated) are attended with q itself.  Every
// (sequence, kv head) is split into n_split ranges of body tiles plus one range for sink +
// residual; each range writes a partial (running max m in log2 units, sum l, output o).  The
// merge kernel combines the partials by log-sum-exp, rotates the body part back with H and
// adds the plain part.
#include "common.hpp"

namespace kvarn {
namespace {

constexpr int kThreads = 256;
constexpr int kPart = 132;  // floats per partial: m, l, 2 pad, o[128]

struct DecodeArgs {
    const uint8_t* k_body;
    const uint8_t* v_body;
    const uint16_t* k_resid;
    const uint16_t* v_resid;
    const uint16_t* k_sink;
    const uint16_t* v_sink;
    const int32_t* seq_len;
    const void* q;
    int q_bf16;
    int n_kv, n_q, g, max_blocks, n_sink, bits;
    float scale_log2;  // sm_scale * log2(e): logits are kept in log2 units
    int n_split, bps;  // body splits per stream and body tiles per split
    float* ws;         // [batch][n_q][n_split + 1][kPart]
};

__device__ __forceinline__ float load_q(const DecodeArgs& a, size_t idx) {
    return a.q_bf16 ? bf16_to_f32(static_cast<const uint16_t*>(a.q)[idx]) : static_cast<const float*>(a.q)[idx];
}

__device__ __forceinline__ float* partial(const DecodeArgs& a, int b, int h, int s) {
    return a.ws + (((size_t)b * a.n_q + h) * (a.n_split + 1) + s) * kPart;
}

// Code e (0..15) of a unit whose words start at w: word e/4/(8/bits), bit 8*(e%4) + bits*((e/4)%(8/bits)).
__device__ __forceinline__ float unit_code(const uint32_t* w, int bits, int e) {
    const int s = e >> 2, q = e & 3;
    if (bits == 2) return (float)((w[0] >> (8 * q + 2 * s)) & 3u);
    return (float)((w[s >> 1] >> (8 * q + 4 * (s & 1))) & 15u);
}

// Per-head reduction of 16 lanes (lanes ^1..^8 of a DPP row).
__device__ __forceinline__ float row16_sum(float v) {
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) v += __shfl_xor(v, m);
    return v;
}
__device__ __forceinline__ float row16_max(float v) {
#pragma unroll
    for (int m = 1; m < 16; m <<= 1) v = fmaxf(v, __shfl_xor(v, m));
    return v;
}

template <int GQ>
struct BodySmem {
    float qrot[GQ][kD];
    float qt[GQ][kD];   // q_rot * a_K of the current tile
    float pt[GQ][kG];   // logits, then p * a_V
    float aux[6][128];  // a_K b_K s2_K a_V b_V s2_V
    float hs[GQ][4];    // per head: running max, running sum, rescale, beta / gamma
};

// Online-softmax update of one tile's logits held in sm.pt (log2 units): per head, new max,
// rescale factor, p (optionally times a_V) back into sm.pt, and returns via sm.hs.
template <int GQ>
__device__ __forceinline__ void softmax_tile(BodySmem<GQ>& sm, int g, int n_valid, const float* aV, const float* bV,
                                             float* m_run, float* l_run) {
    const int tid = threadIdx.x;
    const int j = tid >> 4, part = tid & 15;
    if (j < g) {
        float mx = -INFINITY;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int t = part * 8 + k;
            if (t < n_valid) mx = fmaxf(mx, sm.pt[j][t]);
        }
        mx = row16_max(mx);
        const float m_new = fmaxf(m_run[j], mx);
        const float alpha = m_run[j] == -INFINITY ? 0.f : exp2f(m_run[j] - m_new);
        float lsum = 0.f, gsum = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int t = part * 8 + k;
            float p = 0.f;
            if (t < n_valid) p = exp2f(sm.pt[j][t] - m_new);
            lsum += p;
            if (bV) gsum += p * bV[t];
            sm.pt[j][t] = aV ? p * aV[t] : p;
        }
        lsum = row16_sum(lsum);
        gsum = row16_sum(gsum);
        if (part == 0) {
            sm.hs[j][0] = m_new;
            sm.hs[j][1] = l_run[j] * alpha + lsum;
            sm.hs[j][2] = alpha;
            sm.hs[j][3] = gsum;
        }
    }
    __syncthreads();
    for (int jj = 0; jj < g; ++jj) {
        m_run[jj] = sm.hs[jj][0];
        l_run[jj] = sm.hs[jj][1];
    }
}

template <int GQ>
__device__ void write_partials(const DecodeArgs& a, int b, int kvh, int s, const float* m_run, const float* l_run,
                               const float* o, bool have_o) {
    const int tid = threadIdx.x, c = tid >> 1, hf = tid & 1;
    for (int j = 0; j < a.g; ++j) {
        float* P = partial(a, b, kvh * a.g + j, s);
        if (tid == 0) {
            P[0] = m_run[j];
            P[1] = l_run[j];
        }
        if (hf == 0) P[4 + c] = have_o ? o[j] : 0.f;
    }
}

// One workgroup per (body split, sequence, kv head).
template <int GQ>
__global__ __launch_bounds__(kThreads) void k_decode_body(DecodeArgs a) {
    __shared__ BodySmem<GQ> sm;
    const int tid = threadIdx.x;
    const int split = blockIdx.x % a.n_split;
    const int stream = blockIdx.x / a.n_split;
    const int b = stream / a.n_kv, kvh = stream % a.n_kv;
    const int g = a.g;
    const int len = max(a.seq_len[b], 0);
    // never read past the cache, whatever seq_len holds
    const int nb = min(len > a.n_sink ? (len - a.n_sink) / kG : 0, a.max_blocks);
    const int blk0 = split * a.bps;
    // the last split also takes any tiles beyond the planned range (length above the hint)
    const int blk1 = split == a.n_split - 1 ? nb : min(blk0 + a.bps, nb);

    float m_run[GQ], l_run[GQ], o[GQ];
#pragma unroll
    for (int j = 0; j < GQ; ++j) {
        m_run[j] = -INFINITY;
        l_run[j] = 0.f;
        o[j] = 0.f;
    }
    if (blk0 >= blk1) {
        write_partials<GQ>(a, b, kvh, split, m_run, l_run, o, false);
        return;
    }

    // q of the kv head's query group, rotated: butterflies in LDS
    for (int idx = tid; idx < g * kD; idx += kThreads)
        sm.qrot[idx >> 7][idx & 127] = load_q(a, ((size_t)b * a.n_q + kvh * g) * kD + idx);
    __syncthreads();
    for (int h = 1; h < kD; h <<= 1) {
        for (int idx = tid; idx < g * 64; idx += kThreads) {
            const int j = idx >> 6, r = idx & 63;
            const int i0 = (r / h) * 2 * h + (r % h);
            const float x0 = sm.qrot[j][i0], x1 = sm.qrot[j][i0 + h];
            sm.qrot[j][i0] = x0 + x1;
            sm.qrot[j][i0 + h] = x0 - x1;
        }
        __syncthreads();
    }
    for (int idx = tid; idx < g * kD; idx += kThreads) sm.qrot[idx >> 7][idx & 127] *= kInvSqrt128;
    __syncthreads();

    const size_t tb = tile_bytes(a.bits), cb = code_bytes(a.bits);
    const int words_per_unit = a.bits / 2;
    for (int blk = blk0; blk < blk1; ++blk) {
        const uint8_t* kt = a.k_body + ((size_t)stream * a.max_blocks + blk) * tb;
        const uint8_t* vt = a.v_body + ((size_t)stream * a.max_blocks + blk) * tb;
        if (tid < 192) {
            const int which = tid >> 5, part = tid & 31;
            const uint8_t* base = (which < 3 ? kt : vt) + cb + (which % 3) * 512 + part * 16;
            *reinterpret_cast<float4*>(&sm.aux[which][part * 4]) = *reinterpret_cast<const float4*>(base);
        }
        __syncthreads();
        // q~ = q_rot * a_K and beta = q_rot . b_K per head
        for (int idx = tid; idx < g * kD; idx += kThreads) {
            const int j = idx >> 7, c = idx & 127;
            sm.qt[j][c] = sm.qrot[j][c] * sm.aux[0][c];
        }
        {
            const int j = tid >> 4, part = tid & 15;
            if (j < g) {
                float s = 0.f;
#pragma unroll
                for (int k = 0; k < 8; ++k) s += sm.qrot[j][part * 8 + k] * sm.aux[1][part * 8 + k];
                s = row16_sum(s);
                if (part == 0) sm.hs[j][3] = s;
            }
        }
        __syncthreads();

        // logits: thread (t, half) sums channels 64*half .. 64*half+63 of token t
        {
            const int t = tid >> 1, hf = tid & 1;
            const int sigma = t >> 6, m = t & 15, tau = (t & 63) >> 4;
            float acc[GQ];
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] = 0.f;
            for (int G4 = 0; G4 < 4; ++G4) {
                const int unit = (sigma * 64 + 16 * G4 + m) * 8 + 2 * tau + hf;
                uint32_t w[2];
                w[0] = reinterpret_cast<const uint32_t*>(kt)[unit * words_per_unit];
                w[1] = words_per_unit > 1 ? reinterpret_cast<const uint32_t*>(kt)[unit * words_per_unit + 1] : 0u;
                for (int e = 0; e < 16; ++e) {
                    const float code = unit_code(w, a.bits, e);
                    const int c = 64 * hf + 16 * G4 + e;
#pragma unroll
                    for (int j = 0; j < GQ; ++j)
                        if (j < g) acc[j] += sm.qt[j][c] * code;
                }
            }
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] += __shfl_xor(acc[j], 1);
            if (hf == 0) {
                const float sc = a.scale_log2 * sm.aux[2][t];
#pragma unroll
                for (int j = 0; j < GQ; ++j)
                    if (j < g) sm.pt[j][t] = sc * (acc[j] + sm.hs[j][3]);
            }
        }
        __syncthreads();
        softmax_tile<GQ>(sm, g, kG, sm.aux[3], sm.aux[4], m_run, l_run);

        // values: thread (c, half) sums tokens 64*half .. 64*half+63 of channel c
        {
            const int c = tid >> 1, hf = tid & 1;
            float acc[GQ];
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] = 0.f;
            for (int G4 = 0; G4 < 4; ++G4) {
                const int unit = (hf * 64 + 16 * G4 + (c & 15)) * 8 + (c >> 4);
                uint32_t w[2];
                w[0] = reinterpret_cast<const uint32_t*>(vt)[unit * words_per_unit];
                w[1] = words_per_unit > 1 ? reinterpret_cast<const uint32_t*>(vt)[unit * words_per_unit + 1] : 0u;
                for (int e = 0; e < 16; ++e) {
                    const float code = unit_code(w, a.bits, e);
                    const int t = 64 * hf + 16 * (e >> 2) + 4 * G4 + (e & 3);
#pragma unroll
                    for (int j = 0; j < GQ; ++j)
                        if (j < g) acc[j] += sm.pt[j][t] * code;
                }
            }
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] += __shfl_xor(acc[j], 1);
            if (hf == 0) {
                const float s2 = sm.aux[5][c];
#pragma unroll
                for (int j = 0; j < GQ; ++j)
                    if (j < g) o[j] = o[j] * sm.hs[j][2] + s2 * (acc[j] + sm.hs[j][3]);
            }
        }
        __syncthreads();
    }
    write_partials<GQ>(a, b, kvh, split, m_run, l_run, o, true);
}

// One workgroup per (sequence, kv head): sink + residual tokens, bf16, unrotated.
template <int GQ>
__global__ __launch_bounds__(kThreads) void k_decode_plain(DecodeArgs a) {
    __shared__ BodySmem<GQ> sm;  // qrot holds the unrotated q here
    const int tid = threadIdx.x;
    const int stream = blockIdx.x;
    const int b = stream / a.n_kv, kvh = stream % a.n_kv;
    const int g = a.g;
    const int len = max(a.seq_len[b], 0);
    const int ns = min(len, a.n_sink);
    const int nr = len > a.n_sink ? (len - a.n_sink) % kG : 0;
    const int total = ns + nr;

    float m_run[GQ], l_run[GQ], o[GQ];
#pragma unroll
    for (int j = 0; j < GQ; ++j) {
        m_run[j] = -INFINITY;
        l_run[j] = 0.f;
        o[j] = 0.f;
    }
    if (total == 0) {
        write_partials<GQ>(a, b, kvh, a.n_split, m_run, l_run, o, false);
        return;
    }
    for (int idx = tid; idx < g * kD; idx += kThreads)
        sm.qrot[idx >> 7][idx & 127] = load_q(a, ((size_t)b * a.n_q + kvh * g) * kD + idx);
    __syncthreads();

    auto key_ptr = [&](int tok) -> const uint16_t* {
        return tok < ns ? a.k_sink + ((size_t)stream * a.n_sink + tok) * kD
                        : a.k_resid + ((size_t)stream * kG + (tok - ns)) * kD;
    };
    auto val_ptr = [&](int tok) -> const uint16_t* {
        return tok < ns ? a.v_sink + ((size_t)stream * a.n_sink + tok) * kD
                        : a.v_resid + ((size_t)stream * kG + (tok - ns)) * kD;
    };

    for (int t0 = 0; t0 < total; t0 += kG) {
        const int n = min(kG, total - t0);
        {
            const int t = tid >> 1, hf = tid & 1;
            float acc[GQ];
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] = 0.f;
            if (t < n) {
                const uint16_t* kp = key_ptr(t0 + t) + 64 * hf;
                for (int c = 0; c < 64; ++c) {
                    const float kv = bf16_to_f32(kp[c]);
#pragma unroll
                    for (int j = 0; j < GQ; ++j)
                        if (j < g) acc[j] += sm.qrot[j][64 * hf + c] * kv;
                }
            }
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] += __shfl_xor(acc[j], 1);
            if (hf == 0) {
#pragma unroll
                for (int j = 0; j < GQ; ++j)
                    if (j < g) sm.pt[j][t] = t < n ? a.scale_log2 * acc[j] : -INFINITY;
            }
        }
        __syncthreads();
        softmax_tile<GQ>(sm, g, n, nullptr, nullptr, m_run, l_run);
        {
            const int c = tid >> 1, hf = tid & 1;
            float acc[GQ];
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] = 0.f;
            for (int t = 64 * hf; t < min(n, 64 * hf + 64); ++t) {
                const float vv = bf16_to_f32(val_ptr(t0 + t)[c]);
#pragma unroll
                for (int j = 0; j < GQ; ++j)
                    if (j < g) acc[j] += sm.pt[j][t] * vv;
            }
#pragma unroll
            for (int j = 0; j < GQ; ++j) acc[j] += __shfl_xor(acc[j], 1);
            if (hf == 0) {
#pragma unroll
                for (int j = 0; j < GQ; ++j)
                    if (j < g) o[j] = o[j] * sm.hs[j][2] + acc[j];
            }
        }
        __syncthreads();
    }
    write_partials<GQ>(a, b, kvh, a.n_split, m_run, l_run, o, true);
}

// One 128-thread workgroup per (sequence, query head): log-sum-exp merge of the partials,
// inverse rotation of the body part, normalisation.
__global__ __launch_bounds__(128) void k_decode_merge(DecodeArgs a, void* out, int out_bf16) {
    __shared__ float orot[kD];
    const int c = threadIdx.x;
    const int bh = blockIdx.x;
    const float* P = a.ws + (size_t)bh * (a.n_split + 1) * kPart;
    float M = -INFINITY;
    for (int s = 0; s <= a.n_split; ++s)
        if (P[s * kPart + 1] > 0.f) M = fmaxf(M, P[s * kPart]);
    float L = 0.f, acc = 0.f;
    for (int s = 0; s < a.n_split; ++s) {
        const float l = P[s * kPart + 1];
        if (l > 0.f) {
            const float w = exp2f(P[s * kPart] - M);
            L += w * l;
            acc += w * P[s * kPart + 4 + c];
        }
    }
    orot[c] = acc;
    __syncthreads();
    for (int h = 1; h < kD; h <<= 1) {
        float x0 = 0.f, x1 = 0.f;
        int i0 = 0;
        if (c < 64) {
            i0 = (c / h) * 2 * h + (c % h);
            x0 = orot[i0];
            x1 = orot[i0 + h];
        }
        __syncthreads();
        if (c < 64) {
            orot[i0] = x0 + x1;
            orot[i0 + h] = x0 - x1;
        }
        __syncthreads();
    }
    float o = orot[c] * kInvSqrt128;
    const float* Pp = P + (size_t)a.n_split * kPart;
    if (Pp[1] > 0.f) {
        const float w = exp2f(Pp[0] - M);
        L += w * Pp[1];
        o += w * Pp[4 + c];
    }
    o = L > 0.f ? o / L : 0.f;
    const size_t idx = (size_t)bh * kD + c;
    if (out_bf16)
        static_cast<uint16_t*>(out)[idx] = f32_to_bf16(o);
    else
        static_cast<float*>(out)[idx] = o;
}

template <int GQ>
hipError_t launch_g(const DecodeArgs& a, int batch, void* out, bool out_bf16, hipStream_t stream) {
    const int streams = batch * a.n_kv;
    hipLaunchKernelGGL(k_decode_body<GQ>, dim3((unsigned)(streams * a.n_split)), dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_decode_plain<GQ>, dim3((unsigned)streams), dim3(kThreads), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_decode_merge, dim3((unsigned)(batch * a.n_q)), dim3(128), 0, stream, a, out,
                       out_bf16 ? 1 : 0);
    return hipGetLastError();
}

}  // namespace

DecodePlan plan_decode(int batch, int n_kv, int max_len, int n_sink, int max_blocks) {
    DecodePlan p;
    int nb = max_len > n_sink ? (max_len - n_sink) / kG : 0;
    if (nb > max_blocks) nb = max_blocks;
    p.max_blocks_used = nb;
    const int streams = batch * n_kv;
    // aim for about 2048 workgroups (8 per CU) but never split below one tile
    int want = (2048 + streams - 1) / streams;
    if (want < 1) want = 1;
    if (nb < 1) {
        p.n_split = 1;
        p.blocks_per_split = 1;
        return p;
    }
    if (want > nb) want = nb;
    p.blocks_per_split = (nb + want - 1) / want;
    p.n_split = (nb + p.blocks_per_split - 1) / p.blocks_per_split;
    return p;
}

size_t decode_workspace_bytes(int batch, int n_q, const DecodePlan& plan) {
    return (size_t)batch * n_q * (plan.n_split + 1) * kPart * sizeof(float);
}

hipError_t launch_decode(const kvarn_cache& c, int bits, int n_sink, int n_q, const void* q, bool q_bf16, void* out,
                         bool out_bf16, float sm_scale, const DecodePlan& plan, float* ws, hipStream_t stream) {
    DecodeArgs a;
    a.k_body = static_cast<const uint8_t*>(c.k_body);
    a.v_body = static_cast<const uint8_t*>(c.v_body);
    a.k_resid = static_cast<const uint16_t*>(c.k_resid);
    a.v_resid = static_cast<const uint16_t*>(c.v_resid);
    a.k_sink = static_cast<const uint16_t*>(c.k_sink);
    a.v_sink = static_cast<const uint16_t*>(c.v_sink);
    a.seq_len = c.seq_len;
    a.q = q;
    a.q_bf16 = q_bf16 ? 1 : 0;
    a.n_kv = c.n_kv;
    a.n_q = n_q;
    a.g = n_q / c.n_kv;
    a.max_blocks = c.max_blocks;
    a.n_sink = n_sink;
    a.bits = bits;
    a.scale_log2 = sm_scale * kLog2e;
    a.n_split = plan.n_split;
    a.bps = plan.blocks_per_split;
    a.ws = ws;
    if (a.g <= 1) return launch_g<1>(a, c.batch, out, out_bf16, stream);
    if (a.g <= 2) return launch_g<2>(a, c.batch, out, out_bf16, stream);
    if (a.g <= 4) return launch_g<4>(a, c.batch, out, out_bf16, stream);
    if (a.g <= 8) return launch_g<8>(a, c.batch, out, out_bf16, stream);
    return launch_g<16>(a, c.batch, out, out_bf16, stream);
}

}  // namespace kvarn
