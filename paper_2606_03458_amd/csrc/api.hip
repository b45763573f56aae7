// Host side of the libkvarn C ABI: argument validation (before anything is enqueued), split
// planning and kernel launches.  No device memory is allocated here.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "common.hpp"

using namespace kvarn;

// Split partials of kvarn_decode_attention_noalloc: one array per device, held until the
// process ends.  In host code `scratch` only names the symbol; its device address on the
// current device comes from hipGetSymbolAddress (scratch_ptr below) and is the only form
// passed to kernels.
static __device__ __align__(256) uint8_t scratch[KVARN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's scratch array, looked up once per device.
hipError_t scratch_ptr(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int check_params(const kvarn_params* p) {
    if (!p) return KVARN_EINVAL;
    if (p->bits != 2 && p->bits != 4) return KVARN_EUNSUPPORTED;
    if (p->aux_format != KVARN_AUX_F32 && p->aux_format != KVARN_AUX_COMPACT) return KVARN_EUNSUPPORTED;
    if (p->rotate != 0 && p->rotate != 1) return KVARN_EINVAL;
    if (p->varn_iters < 0 || p->varn_iters > 64) return KVARN_EINVAL;
    if (p->n_sink < 0 || p->n_sink > 1024) return KVARN_EINVAL;
    // ranges that keep exp(+-L) and log(v) of the quantizer inside the normal fp32 range
    if (!(p->var_min >= 1e-30f) || !(p->var_max <= 1e30f) || p->var_min > p->var_max) return KVARN_EINVAL;
    if (!(p->log_lo >= -40.f) || !(p->log_hi <= 40.f) || p->log_lo > p->log_hi) return KVARN_EINVAL;
    return KVARN_OK;
}

// Arguments of an append; *flush: whether the call has to launch the flush (always without the
// length hint, else when the token fills the residual).
int append_check(const kvarn_params* p, const kvarn_cache* cache, const void* k_new, const void* v_new, int32_t dtype,
                 int32_t host_len_before, bool* flush);

QParams qparams(const kvarn_params* p) {
    return QParams{p->bits, p->varn_iters, p->var_min, p->var_max, p->log_lo, p->log_hi,
                   p->aux_format == KVARN_AUX_COMPACT ? 1 : 0, p->rotate};
}

int check_cache(const kvarn_params* p, const kvarn_cache* c) {
    if (!c) return KVARN_EINVAL;
    if (c->batch <= 0 || c->n_kv <= 0 || c->max_blocks < 0) return KVARN_EINVAL;
    // kernels index (sequence, kv head, K|V) in 32 bits
    if ((int64_t)c->batch * c->n_kv > kMaxStreams) return KVARN_EINVAL;
    if (!c->k_body || !c->v_body || !c->k_resid || !c->v_resid || !c->seq_len) return KVARN_EINVAL;
    if (p->n_sink > 0 && (!c->k_sink || !c->v_sink)) return KVARN_EINVAL;
    if (!aligned(c->k_body, 16) || !aligned(c->v_body, 16) || !aligned(c->k_resid, 16) || !aligned(c->v_resid, 16))
        return KVARN_EINVAL;
    if (p->n_sink > 0 && (!aligned(c->k_sink, 16) || !aligned(c->v_sink, 16))) return KVARN_EINVAL;
    if (!aligned(c->seq_len, 4)) return KVARN_EINVAL;
    if (c->block_table && (c->n_phys <= 0 || !aligned(c->block_table, 4))) return KVARN_EINVAL;
    return KVARN_OK;
}

int check_dtype(int32_t d) { return (d == KVARN_F32 || d == KVARN_BF16) ? KVARN_OK : KVARN_EINVAL; }

int append_check(const kvarn_params* p, const kvarn_cache* cache, const void* k_new, const void* v_new, int32_t dtype,
                 int32_t host_len_before, bool* flush) {
    int st = check_params(p);
    if (st) return st;
    st = check_cache(p, cache);
    if (st) return st;
    if (check_dtype(dtype)) return KVARN_EINVAL;
    if (!k_new || !v_new) return KVARN_EINVAL;
    const size_t va = dtype == KVARN_BF16 ? 8 : 16;
    if (!aligned(k_new, va) || !aligned(v_new, va)) return KVARN_EINVAL;
    if (host_len_before < -1) return KVARN_EINVAL;
    *flush = true;
    if (host_len_before >= 0) {
        const int len = host_len_before;
        *flush = false;
        if (len >= p->n_sink) {
            const int r = (len - p->n_sink) % kG, nb = (len - p->n_sink) / kG;
            if (r == kG - 1) {
                if (nb >= cache->max_blocks) return KVARN_ECAPACITY;
                *flush = true;
            }
        }
    }
    return KVARN_OK;
}

}  // namespace

extern "C" {

int kvarn_params_init(kvarn_params* p, int32_t bits) {
    if (!p) return KVARN_EINVAL;
    if (bits != 2 && bits != 4) return KVARN_EUNSUPPORTED;
    p->bits = bits;
    p->varn_iters = 8;
    p->n_sink = 0;
    p->var_min = 1e-8f;
    p->var_max = 1e8f;
    p->log_lo = -0.3f;
    p->log_hi = 10.0f;
    p->aux_format = KVARN_AUX_F32;
    p->rotate = 1;
    return KVARN_OK;
}

size_t kvarn_tile_bytes(const kvarn_params* p) {
    return check_params(p) ? 0 : tile_bytes(p->bits, p->aux_format == KVARN_AUX_COMPACT);
}

int kvarn_cache_sizes(const kvarn_params* p, int32_t batch, int32_t n_kv, int32_t max_blocks, size_t sizes[7]) {
    int st = check_params(p);
    if (st) return st;
    if (!sizes || batch <= 0 || n_kv <= 0 || max_blocks < 0) return KVARN_EINVAL;
    if ((int64_t)batch * n_kv > kMaxStreams) return KVARN_EINVAL;
    const size_t streams = (size_t)batch * n_kv;
    sizes[0] = sizes[1] = streams * max_blocks * tile_bytes(p->bits, p->aux_format == KVARN_AUX_COMPACT);
    sizes[2] = sizes[3] = streams * kG * kD * sizeof(uint16_t);
    sizes[4] = sizes[5] = streams * (size_t)p->n_sink * kD * sizeof(uint16_t);
    sizes[6] = (size_t)batch * sizeof(int32_t);
    return KVARN_OK;
}

int kvarn_quantize_block(const kvarn_params* p, int32_t kind, const void* x, int32_t x_dtype, int64_t n_outer,
                         int64_t n_inner, int64_t x_outer_stride, int64_t x_inner_stride, int64_t x_token_stride,
                         void* out, int64_t out_outer_stride, int64_t out_inner_stride, int32_t* best_iter,
                         hipStream_t stream) {
    int st = check_params(p);
    if (st) return st;
    if (kind != KVARN_KEYS && kind != KVARN_VALUES) return KVARN_EINVAL;
    if (check_dtype(x_dtype)) return KVARN_EINVAL;
    if (n_outer < 0 || n_inner < 0 || x_outer_stride < 0 || x_inner_stride < 0 || x_token_stride < 0 ||
        out_outer_stride < 0 || out_inner_stride < 0)
        return KVARN_EINVAL;
    if (n_outer == 0 || n_inner == 0) return KVARN_OK;
    if (!x || !out) return KVARN_EINVAL;
    const int64_t esz = x_dtype == KVARN_BF16 ? 2 : 4;
    // rows are read as 16-byte vectors
    if (!aligned(x, 16) || (x_token_stride * esz) % 16 || (x_outer_stride * esz) % 16 || (x_inner_stride * esz) % 16)
        return KVARN_EINVAL;
    if (x_token_stride < kD) return KVARN_EINVAL;  // tokens must not overlap
    if (!aligned(out, 16)) return KVARN_EINVAL;
    if (best_iter && !aligned(best_iter, 4)) return KVARN_EINVAL;
    hipError_t e = launch_quantize_tiles(qparams(p), kind, x, x_dtype == KVARN_BF16, n_outer, n_inner, x_outer_stride,
                                         x_inner_stride, x_token_stride, out, out_outer_stride, out_inner_stride,
                                         best_iter, stream);
    return e == hipSuccess ? KVARN_OK : KVARN_EHIP;
}

int kvarn_append_token(const kvarn_params* p, const kvarn_cache* cache, const void* k_new, const void* v_new,
                       int32_t dtype, int32_t host_len_before, hipStream_t stream) {
    bool flush = true;
    const int st = append_check(p, cache, k_new, v_new, dtype, host_len_before, &flush);
    if (st) return st;
    hipError_t e = launch_append(*cache, p->n_sink, k_new, v_new, dtype == KVARN_BF16, stream);
    if (e != hipSuccess) return KVARN_EHIP;
    if (flush) {
        e = launch_flush(qparams(p), *cache, p->n_sink, host_len_before >= 0, stream);
        if (e != hipSuccess) return KVARN_EHIP;
    }
    return KVARN_OK;
}

int kvarn_prefill(const kvarn_params* p, const kvarn_cache* cache, const void* k, const void* v, int32_t dtype,
                  const int32_t* cu_seqlens, int32_t max_len, hipStream_t stream) {
    int st = check_params(p);
    if (st) return st;
    st = check_cache(p, cache);
    if (st) return st;
    if (check_dtype(dtype)) return KVARN_EINVAL;
    if (!k || !v || !cu_seqlens || max_len < 0) return KVARN_EINVAL;
    if (!aligned(k, 16) || !aligned(v, 16) || !aligned(cu_seqlens, 4)) return KVARN_EINVAL;
    const hipError_t e = launch_prefill(qparams(p), *cache, p->n_sink, k, v, dtype == KVARN_BF16, cu_seqlens, max_len,
                                        stream);
    return e == hipSuccess ? KVARN_OK : KVARN_EHIP;
}

size_t kvarn_decode_workspace_bytes(const kvarn_params* p, const kvarn_cache* cache, int32_t n_q,
                                    int32_t max_len_hint) {
    if (check_params(p) || !cache || cache->batch <= 0 || cache->n_kv <= 0 || n_q <= 0 || max_len_hint < 0) return 0;
    const DecodePlan plan = plan_decode(cache->batch, cache->n_kv, n_q, p->bits, max_len_hint, p->n_sink, cache->max_blocks);
    return decode_workspace_bytes(cache->batch, n_q, plan);
}

}  // extern "C"

namespace {

// Validation and planning shared by the decode entry points; nothing is enqueued.  ws == nullptr
// with use_scratch: the partials go to the library's per-device scratch array (*workspace is set
// to it).
int decode_check(const kvarn_params* p, const kvarn_cache* cache, int32_t n_q, const void* q, int32_t q_dtype,
                 const void* out, int32_t out_dtype, float sm_scale, int32_t max_len_hint, void** workspace,
                 size_t workspace_bytes, bool use_scratch, DecodePlan* plan) {
    int st = check_params(p);
    if (st) return st;
    st = check_cache(p, cache);
    if (st) return st;
    if (n_q <= 0 || n_q % cache->n_kv != 0 || n_q / cache->n_kv > 16) return KVARN_EINVAL;
    if (check_dtype(q_dtype) || check_dtype(out_dtype)) return KVARN_EINVAL;
    if (!q || !out || !std::isfinite(sm_scale) || max_len_hint < 0) return KVARN_EINVAL;
    if (!aligned(q, 4) || !aligned(out, 8)) return KVARN_EINVAL;
    *plan = plan_decode(cache->batch, cache->n_kv, n_q, p->bits, max_len_hint, p->n_sink, cache->max_blocks);
    const size_t need = decode_workspace_bytes(cache->batch, n_q, *plan);
    if (use_scratch) {
        if (need > KVARN_NOALLOC_SCRATCH_BYTES) return KVARN_EWORKSPACE;
        *workspace = nullptr;
        if (need > 0 && scratch_ptr(workspace) != hipSuccess) return KVARN_EHIP;
    } else if (need > 0 && (!*workspace || workspace_bytes < need || !aligned(*workspace, 16))) {
        return KVARN_EWORKSPACE;
    }
    return KVARN_OK;
}

int decode_launch(const kvarn_params* p, const kvarn_cache* cache, int32_t n_q, const void* q, int32_t q_dtype,
                  void* out, int32_t out_dtype, float sm_scale, const DecodePlan& plan, void* workspace,
                  hipStream_t stream, const StepAppend* step = nullptr) {
    const hipError_t e = launch_decode(*cache, p->bits, p->aux_format == KVARN_AUX_COMPACT, p->rotate, p->n_sink, n_q,
                                       q, q_dtype == KVARN_BF16, out, out_dtype == KVARN_BF16, sm_scale, plan,
                                       static_cast<float*>(workspace), stream, step);
    return e == hipSuccess ? KVARN_OK : KVARN_EHIP;
}

int decode_impl(const kvarn_params* p, const kvarn_cache* cache, int32_t n_q, const void* q, int32_t q_dtype,
                void* out, int32_t out_dtype, float sm_scale, int32_t max_len_hint, void* workspace,
                size_t workspace_bytes, bool use_scratch, hipStream_t stream) {
    DecodePlan plan;
    const int st = decode_check(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, max_len_hint, &workspace,
                                workspace_bytes, use_scratch, &plan);
    if (st) return st;
    return decode_launch(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, plan, workspace, stream);
}

}  // namespace

extern "C" {

int kvarn_decode_attention(const kvarn_params* p, const kvarn_cache* cache, int32_t n_q, const void* q,
                           int32_t q_dtype, void* out, int32_t out_dtype, float sm_scale, int32_t max_len_hint,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return decode_impl(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, max_len_hint, workspace, workspace_bytes,
                       false, stream);
}

int kvarn_decode_attention_noalloc(const kvarn_params* p, const kvarn_cache* cache, int32_t n_q, const void* q,
                                   int32_t q_dtype, void* out, int32_t out_dtype, float sm_scale,
                                   int32_t max_len_hint, hipStream_t stream) {
    return decode_impl(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, max_len_hint, nullptr, 0, true, stream);
}

int kvarn_append_decode(const kvarn_params* p, const kvarn_cache* cache, const void* k_new, const void* v_new,
                        int32_t kv_dtype, int32_t host_len_before, int32_t n_q, const void* q, int32_t q_dtype,
                        void* out, int32_t out_dtype, float sm_scale, void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
    if (host_len_before < 0 || host_len_before == INT32_MAX) return KVARN_EINVAL;
    bool flush = true;
    int st = append_check(p, cache, k_new, v_new, kv_dtype, host_len_before, &flush);
    if (st) return st;
    DecodePlan plan;
    st = decode_check(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, host_len_before + 1, &workspace,
                      workspace_bytes, false, &plan);
    if (st) return st;
    if (kv_dtype == KVARN_BF16 && host_len_before >= p->n_sink && !flush && aligned(k_new, 16) && aligned(v_new, 16)) {
        const StepAppend step{host_len_before, k_new, v_new};
        return decode_launch(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, plan, workspace, stream, &step);
    }
    hipError_t e = launch_append(*cache, p->n_sink, k_new, v_new, kv_dtype == KVARN_BF16, stream);
    if (e == hipSuccess && flush) e = launch_flush(qparams(p), *cache, p->n_sink, true, stream);
    if (e != hipSuccess) return KVARN_EHIP;
    return decode_launch(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale, plan, workspace, stream);
}

}  // extern "C"
