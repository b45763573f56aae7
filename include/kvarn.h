/*
 * kvarn.h -- C ABI of libkvarn, the KVarN hot path for AMD Instinct MI355X (gfx950).
 *
 * KVarN (arXiv 2606.03458) stores a transformer's K/V cache in three regions (App. D,
 * "Quantization"): the first n_sink tokens of a sequence in 16-bit, a body of quantized
 * 128-token groups, and a residual of the most recent tokens that do not yet fill a group.
 * A group (one 128-token x 128-channel tile of K or of V for one sequence and kv head) is
 * quantized by (Fig. 2, Sec. 3.3):
 *   1. a Hadamard rotation of every token along head_dim (Sec. 2.2, App. A),
 *   2. VarN, alternating log-domain variance normalisation of columns and rows with best-
 *      imbalance tracking (App. H, Algorithm 1; rows = tokens, columns = channels),
 *   3. asymmetric round-to-nearest (Sec. 2.1, Eq. 1): keys per channel, values per token,
 *   4. dual-scale storage with the Sinkhorn scale of the group axis absorbed into the RTN
 *      scale and offset (App. D, "Effective memory overhead").
 * Decode attention reads the packed body, dequantizes with the second scale fused (App. I)
 * and attends over sink + body + residual.
 *
 * Conventions for every entry point:
 *   - All pointers to tensors are DEVICE pointers, owned by the caller, and must stay valid
 *     until the work queued on `stream` has run.  The library allocates no device memory at
 *     run time; its code object holds one static scratch array per device, used only by
 *     kvarn_decode_attention_noalloc.
 *   - Every call only enqueues work on `stream` (asynchronous); none synchronizes.
 *   - Arguments are validated on the host before anything is enqueued.  A failed check
 *     returns a negative kvarn_status and enqueues nothing.  KVARN_EHIP reports a failed
 *     kernel launch.  The library never aborts and throws nothing across this ABI.
 *   - Calls on different caches may run concurrently; calls that touch the same cache must
 *     be ordered by the caller (same stream or events).
 *   - head_dim and the group size are fixed at 128.
 *
 * Packed tile (the library's storage format; the paper fixes only what is stored per group):
 *   bytes [0, bits*2048)          128 x 128 codes of `bits` bits (layout below)
 *   then the aux, in one of two formats (kvarn_params.aux_format):
 *   KVARN_AUX_F32:
 *     512 bytes   a[128]  fp32   keys: RTN scale of channel c times its Sinkhorn channel
 *                                scale; values: of token t
 *     512 bytes   b[128]  fp32   the matching offset (group minimum times the same scale)
 *     512 bytes   s2[128] fp32   second scale: keys per token, values per channel (the other
 *                                Sinkhorn scale)
 *     Tile size 5632 bytes at 2 bits (2.75 bits/element), 9728 at 4 bits.
 *   KVARN_AUX_COMPACT (App. D, "Effective memory overhead": per group of 128 values, both
 *   scales in an 8-bit float format and the zero point in a 16-bit one):
 *     256 bytes   b[128]  IEEE binary16, little-endian
 *     128 bytes   a[128]  OCP E4M3 (4-bit exponent, bias 7, 3-bit mantissa, largest 448)
 *     128 bytes   s2[128] OCP E4M3
 *     s2 is rounded to nearest first and the tile is quantized against the stored s2; a is the
 *     RTN step rounded upward (the stored range covers the group), b the nearest binary16 of
 *     the group minimum, and codes are chosen for the stored a and b.  Scales are kept within
 *     [2^-6, 448] and b within +-65504.  When the largest step of a tile exceeds 448, a
 *     tile-wide power of two 2^e moves from a and b into s2 (the smallest e that fits, as far
 *     as the largest s2 stays within 448; only when no other-axis scale is below 2^-6), which
 *     leaves every dequantized value unchanged.  Tile size 4608 bytes at 2 bits (2.25 bits/element),
 *     8704 at 4 bits.
 *   Dequantized rotated tile, both formats: keys (code[t][c]*a[c] + b[c]) * s2[t]; values
 *   (code[t][c]*a[t] + b[t]) * s2[c]; un-rotate each token with the orthonormal Hadamard
 *   matrix.
 *   Code layout: codes form units of 16; a unit is bits/2 little-endian 32-bit words.  With
 *   u = 512*sigma + 8*L + w (L in 0..63, w in 0..7) and p = 8/bits, unit u starts at word
 *   512*(bits/2)*sigma + 256*(w/p) + 4*L + (bits/2)*(w%p).  Code e = 4*s + q (s, q in 0..3)
 *   of a unit sits in word s/p of the unit, at bit 8*q + bits*(s%p).  For token t, channel c,
 *   sigma = t/64:
 *     keys:   u = (sigma*64 + 16*((c%64)/16) + t%16)*8 + 2*((t%64)/16) + c/64,  e = c % 16
 *     values: u = (sigma*64 + 16*((t%16)/4) + c%16)*8 + c/16,  e = 4*((t%64)/16) + t%4
 *   (Each 64-token half of a tile is the register image of 64 GPU lanes x 8 units: lane L
 *   holds units 8L .. 8L+7 as 2 or 4 pieces of 16 bytes, piece k at byte 1024*k + 16*L of
 *   the half, so that each 16-byte load of a wave reads 1 KB of consecutive bytes.)
 */
#ifndef KVARN_H
#define KVARN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVARN_API __attribute__((visibility("default")))

typedef enum {
    KVARN_OK = 0,
    KVARN_EINVAL = -1,       /* null pointer, bad size, stride or dtype                      */
    KVARN_EUNSUPPORTED = -2, /* valid request the library does not implement (e.g. bits=3)  */
    KVARN_ECAPACITY = -3,    /* the cache has no room for the requested tokens              */
    KVARN_EHIP = -4,         /* a HIP launch or query failed                                */
    KVARN_EWORKSPACE = -5    /* workspace missing or smaller than kvarn_decode_workspace_bytes */
} kvarn_status;

typedef enum { KVARN_F32 = 0, KVARN_BF16 = 1 } kvarn_dtype;
typedef enum { KVARN_KEYS = 0, KVARN_VALUES = 1 } kvarn_kind;

/* Quantizer constants (App. H, Algorithm 1).  kvarn_params_init fills the defaults. */
typedef struct {
    int32_t bits;       /* 2 or 4                                                      */
    int32_t varn_iters; /* K of Algorithm 1: 8 (runtime experiment, Sec. 4.2); 0..64      */
    int32_t n_sink;     /* tokens kept in bf16 at the start of a sequence: 0 or up to 1024 */
    float var_min;      /* c_min: variances are clamped to [var_min, var_max]; 1e-8     */
    float var_max;      /* c_max: 1e8 (the paper gives no values for c_min, c_max)      */
    float log_lo;       /* clamp of the cumulative log-scales: -0.3 (Algorithm 1)       */
    float log_hi;       /* 10.0 (Algorithm 1)                                           */
    int32_t aux_format; /* KVARN_AUX_F32 (default) or KVARN_AUX_COMPACT                  */
    int32_t rotate;     /* 1 (default): Hadamard rotation before VarN, as KVarN does.  0: no
                         * rotation -- with varn_iters = 0 the quantizer is KIVI-style RTN,
                         * with varn_iters > 0 VarN alone (the ablations of Fig. 1).  Tiles
                         * then hold the unrotated domain and decode skips both rotations;
                         * every call on one cache must use the same value. */
} kvarn_params;
typedef enum { KVARN_AUX_F32 = 0, KVARN_AUX_COMPACT = 1 } kvarn_aux_format;
/* Accepted ranges (else KVARN_EINVAL): 1e-30 <= var_min <= var_max <= 1e30 and
 * -40 <= log_lo <= log_hi <= 40, which keeps every scale exp(+-L) and every log of a clamped
 * variance inside the normal fp32 range. */

/* The cache of `batch` sequences with n_kv kv heads each (a model's layers may be folded
 * into batch; batch * n_kv at most 2^26, else KVARN_EINVAL).  Device buffers, all
 * caller-allocated (sizes from kvarn_cache_sizes):
 *   k_body, v_body   [batch][n_kv][max_blocks] packed tiles of kvarn_tile_bytes(p)
 *   k_resid, v_resid [batch][n_kv][128][128]    bf16, tokens as given (unrotated)
 *   k_sink, v_sink   [batch][n_kv][n_sink][128] bf16, or NULL when n_sink == 0
 *   seq_len          [batch] int32: tokens held by each sequence (all regions)
 *   err_word         one uint32 or NULL: a kernel that finds no room sets bit 0 and drops
 *                    the write instead of writing out of bounds (a backstop only: the host
 *                    check of kvarn_append_token catches overflow from its length hint); an
 *                    invalid block id (below) sets bit 1; a fused append step over a
 *                    sequence whose length is not the host's (kvarn_append_decode) sets bit 2.
 *   block_table      NULL for the dense body above.  Otherwise the paged layout of serving
 *                    engines: block_table is [batch][max_blocks] int32 on the device and
 *                    k_body, v_body are pools of n_phys blocks, [n_phys][n_kv] tiles each;
 *                    body tile blk of (sequence b, kv head h) is tile h of pool block
 *                    block_table[b][blk].  Only the entries of tiles a call touches are read.
 *                    An id outside [0, n_phys) sets bit 1 of err_word; decode then skips the
 *                    sequence's body and flush / prefill do not write the tile.
 *   n_phys           pool size in blocks, when block_table is set (pool bytes: n_phys * n_kv *
 *                    kvarn_tile_bytes(p) for each of k_body and v_body).
 * A sequence of length L holds min(L, n_sink) sink tokens, (L - n_sink)/128 body tiles and
 * (L - n_sink) % 128 residual tokens (0 body and residual tokens while L <= n_sink). */
typedef struct {
    int32_t batch, n_kv, max_blocks;
    void *k_body, *v_body;
    void *k_resid, *v_resid;
    void *k_sink, *v_sink;
    int32_t *seq_len;
    uint32_t *err_word;
    const int32_t *block_table;
    int32_t n_phys;
} kvarn_cache;

/* Fill `p` with the defaults for `bits` (2 or 4; fp32 aux).  Returns KVARN_EINVAL for a null
 * `p`, KVARN_EUNSUPPORTED for other bit widths. */
KVARN_API int kvarn_params_init(kvarn_params *p, int32_t bits);

/* Bytes of one packed tile for p's bits and aux format (5632 / 9728 with fp32 aux, 4608 / 8704
 * compact); 0 for invalid parameters. */
KVARN_API size_t kvarn_tile_bytes(const kvarn_params *p);

/* Byte sizes of the seven cache buffers, in the order k_body, v_body, k_resid, v_resid,
 * k_sink, v_sink, seq_len.  Returns KVARN_EINVAL for null pointers or non-positive sizes. */
KVARN_API int kvarn_cache_sizes(const kvarn_params *p, int32_t batch, int32_t n_kv, int32_t max_blocks, size_t sizes[7]);

/*
 * Quantize n_outer x n_inner independent tiles (Fig. 2: Hadamard, VarN, RTN, pack).
 *   kind    KVARN_KEYS (RTN per channel) or KVARN_VALUES (RTN per token)
 *   x       tile (i, j) starts at element x + i*x_outer_stride + j*x_inner_stride; token t of
 *           it at + t*x_token_stride; its 128 channels are contiguous.  dtype fp32 or bf16.
 *           The input is unrotated: the library applies the Hadamard rotation.
 *   out     tile (i, j) is written at byte out + (i*out_outer_stride + j*out_inner_stride) *
 *           kvarn_tile_bytes(p) (strides counted in tiles).
 *   best_iter  optional [n_outer*n_inner] int32 (row-major over (i, j)): the VarN iteration
 *           whose scales were kept (0 = the initial unit scales); NULL to skip.
 * Strides must be non-negative, x_token_stride >= 128; x, and every x stride times the
 * element size, must be multiples of 16 bytes (rows are read as 16-byte vectors); out must
 * be 16-byte aligned.  n_outer or n_inner == 0 is a no-op.
 * Prefill: quantize [batch*n_kv][T/128] tiles straight into k_body / v_body and set seq_len.
 */
KVARN_API int kvarn_quantize_block(const kvarn_params *p, int32_t kind, const void *x, int32_t x_dtype, int64_t n_outer,
                         int64_t n_inner, int64_t x_outer_stride, int64_t x_inner_stride, int64_t x_token_stride,
                         void *out, int64_t out_outer_stride, int64_t out_inner_stride, int32_t *best_iter,
                         hipStream_t stream);

/*
 * Prefill whole prompts of different lengths in one call (the bulk write before decode):
 *   k, v        [total_tokens][n_kv][128] in `dtype` (fp32 or bf16), unrotated, 16-byte
 *               aligned; sequence b owns rows cu_seqlens[b] .. cu_seqlens[b+1] - 1
 *   cu_seqlens  [batch + 1] int32 on the device: row offsets, non-decreasing, cu_seqlens[0] = 0
 *   max_len     host bound on the prompt lengths; it sizes the launch
 * Each sequence's contents are replaced by its prompt of length L: seq_len[b] = L, the first
 * min(L, n_sink) tokens go to the sink, every full 128-token group after them is quantized
 * (Fig. 2) into body tiles 0, 1, ... (through block_table when paged), and the remaining
 * (L - n_sink) % 128 tokens go to the residual, as the same tokens appended one by one would
 * leave them.  Sink and residual are stored as bf16.  A sequence with L > max_len or needing
 * more than max_blocks tiles is not written: its seq_len is set to 0 and bit 0 of err_word is
 * set.  Returns KVARN_EINVAL for null or misaligned pointers, a bad dtype or max_len < 0.
 */
KVARN_API int kvarn_prefill(const kvarn_params *p, const kvarn_cache *cache, const void *k, const void *v,
                            int32_t dtype, const int32_t *cu_seqlens, int32_t max_len, hipStream_t stream);

/*
 * Append one token to every (sequence, kv head) (the streaming write of Fig. 4's pseudo-decode):
 *   k_new, v_new  [batch][n_kv][128] in `dtype` (fp32 or bf16; stored as bf16, unrotated).
 * The token goes to the sink while a sequence is shorter than n_sink, otherwise to the
 * residual; a residual that reaches 128 tokens is quantized (keys and values) into the next
 * body tile and emptied, within this call.  seq_len is incremented on the device.
 *   host_len_before  the common length of all sequences before this call (lock-step decode),
 *           used to check capacity on the host and to launch the flush only when one is due;
 *           pass -1 if lengths differ or are unknown: the flush kernel then runs every call
 *           on a grid of resident size (768 workgroups) whose workgroups check the tiles in
 *           turn, each sequence deciding on the device, and overflow is caught by err_word only.
 * Returns KVARN_ECAPACITY (enqueuing nothing) if the hint shows that a flush would need body
 * tile max_blocks.
 */
KVARN_API int kvarn_append_token(const kvarn_params *p, const kvarn_cache *cache, const void *k_new, const void *v_new,
                       int32_t dtype, int32_t host_len_before, hipStream_t stream);

/* Workspace bytes that kvarn_decode_attention needs for these sizes (split partials); 0 when
 * the plan keeps every (sequence, kv head) in one split or in a few splits merged inside one
 * workgroup, or when an argument is invalid. */
KVARN_API size_t kvarn_decode_workspace_bytes(const kvarn_params *p, const kvarn_cache *cache, int32_t n_q,
                                    int32_t max_len_hint);

/*
 * Decode attention of one query token per sequence over its whole cache:
 *   out[b][h][:] = softmax(sm_scale * q[b][h] . K^T) V over the sink, body and residual of
 *   sequence b, kv head h / (n_q / n_kv).  The body is dequantized in registers with both
 *   scales fused (App. I); the query is rotated once so body logits are computed in the
 *   rotated domain, and the body's output is rotated back once per query head (App. A).
 *   q    [batch][n_q][128] fp32 or bf16 (post-RoPE, unrotated)
 *   out  [batch][n_q][128] in out_dtype (fp32 or bf16)
 *   max_len_hint  an upper bound of every seq_len (sizes the split-K plan)
 *   workspace  device buffer of at least kvarn_decode_workspace_bytes(...) bytes, 16-byte
 *           aligned; may be NULL when that size is 0
 * n_q must be a positive multiple of n_kv with n_q / n_kv <= 16; q 4-byte and out 8-byte
 * aligned.  A sequence of length 0 produces zeros.
 */
KVARN_API int kvarn_decode_attention(const kvarn_params *p, const kvarn_cache *cache, int32_t n_q, const void *q,
                           int32_t q_dtype, void *out, int32_t out_dtype, float sm_scale, int32_t max_len_hint,
                           void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * One decode step of a lock-step batch (Fig. 4: each generated token is appended to the cache,
 * then attended over it, new token included; App. D three-region cache): the results of
 * kvarn_append_token(p, cache, k_new, v_new, kv_dtype, host_len_before) followed by
 * kvarn_decode_attention(p, cache, n_q, q, q_dtype, out, out_dtype, sm_scale,
 * host_len_before + 1, workspace, workspace_bytes), bit for bit, in cache and output.
 *   host_len_before  required: the length of every sequence before the call (seq_len on the
 *           device must hold it).
 *   workspace  as for kvarn_decode_attention with max_len_hint = host_len_before + 1.
 * When the token goes to the residual without filling it, is bf16 and k_new, v_new are 16-byte
 * aligned, the append runs inside the decode launch: the wave that attends the residual's last
 * chunk reads the new row from k_new / v_new and stores it into the residual, and seq_len is
 * set to host_len_before + 1 without the decode reading it; one launch instead of two.  A
 * sequence whose seq_len is not host_len_before is then left unchanged and bit 2 of err_word
 * is set (its output is not meaningful).  Otherwise (a sink token, a flush, fp32 tokens) the
 * call runs the two entry points' kernels in turn.
 * Errors: those of both entry points, all checked before anything is enqueued; KVARN_EINVAL for
 * host_len_before < 0 or = INT32_MAX.
 */
KVARN_API int kvarn_append_decode(const kvarn_params *p, const kvarn_cache *cache, const void *k_new,
                                  const void *v_new, int32_t kv_dtype, int32_t host_len_before, int32_t n_q,
                                  const void *q, int32_t q_dtype, void *out, int32_t out_dtype, float sm_scale,
                                  void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Decode attention that allocates nothing, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Arguments and results are those of kvarn_decode_attention without the workspace: the split
 * partials go to a scratch array of KVARN_NOALLOC_SCRATCH_BYTES (32 MiB) that the library
 * holds in static device memory, one array per device, kept until the process ends.  Its
 * device address is looked up once per device (hipGetSymbolAddress, on the first call with
 * that device current, guarded by a mutex); no call allocates or frees anything.
 *   - Plans whose partials need more than KVARN_NOALLOC_SCRATCH_BYTES (as
 *     kvarn_decode_workspace_bytes reports) return KVARN_EWORKSPACE and enqueue nothing.
 *   - Every call on one device shares that device's array: calls that may overlap on one
 *     device (other streams, other host threads) race on it and must be ordered by the
 *     caller.  The array keeps the last call's partials; no call relies on its contents.
 */
#define KVARN_NOALLOC_SCRATCH_BYTES (32u << 20)
KVARN_API int kvarn_decode_attention_noalloc(const kvarn_params *p, const kvarn_cache *cache, int32_t n_q,
                                             const void *q, int32_t q_dtype, void *out, int32_t out_dtype,
                                             float sm_scale, int32_t max_len_hint, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* KVARN_H */
