// KVarN decode attention for gfx950 (App. D three-region cache, App. I fused second scale,
// App. A rotation layout).
//
// Body tiles are attended in the rotated domain.  With q_rot = H q and a tile's aux
//   logit[t]  = s2K[t] * (sum_c q~[c] code[t][c] + beta),   q~ = q_rot * a_K, beta = q_rot . b_K
//   o_rot[c] += s2V[c] * (sum_t p~[t] code[t][c] + gamma),  p~ = p * a_V,   gamma = p . b_V
// so both dual-scale products are fused into one pass over the codes (App. I).
//
// The two sums over codes are matrix products on the int8 matrix cores
// (v_mfma_i32_16x16x64_i8).  The codes are exact int8 operands taken straight from the packed
// words (the tile format stores them in the MFMA register order).  The real-valued side is
// written as a fixed-point integer split into signed base-256 digits, recombined exactly in
// int32.  Integer accumulation is exact, so the only rounding in the code terms is that of q~
// and p~ to their fixed-point grids.
//
// The digits of a head are rows of one MFMA operand (three digits for both q~ and p~: 22 bits
// at 2-bit codes, 20 at 4-bit), and beta, gamma are plain fp32 dot products of the unrounded
// q_rot and p with the offsets.  A wave takes up to eight query heads of a kv head's group (one
// or two head groups of four, or four plus a fifth carried in the empty digit slots); larger
// groups are taken in chunks of at most eight heads, one wave per chunk.
//
// Sink and residual tokens (bf16, unrotated) use the bf16 matrix cores for q . k (q as a bf16
// pair hi + lo when it is fp32) and plain FMAs for p . v, in chunks of 32 tokens.  One wave owns
// a (split, sequence, kv head, head chunk).  An unsplit stream's one wave takes sink + residual
// after its body tiles; a split stream's sink and residual chunks get splits of their own (one
// per chunk when the waves fit), which run beside the body splits, or the body splits share
// them.  A single split writes the final output directly (inverse rotation in LDS); up to four
// splits of a stream are the waves of one workgroup and combine by log-sum-exp through LDS
// before writing it; more write partials that the merge kernel combines.
//
// A lock-step decode step can append its token in the same launch (Fig. 4): the new row is the
// residual's last, read from the token input by the wave that attends that chunk, which also
// stores it into the residual; the step's length comes from the host.
#include <algorithm>

#include "common.hpp"

namespace kvarn {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));

constexpr int kPart = 260;  // floats per partial: m, l, 2 pad, o_rot[128], o_plain[128]
constexpr int kRC = 32;     // bf16 tokens (sink / residual) per chunk
// splits of a stream that may form one workgroup (one wave per SIMD; groups of 5-6 waves
// measured slower than the separate merge on the 2-bit streaming runs)
constexpr int kMaxGroup = 4;
// body tiles below which a stream planned with at most kMaxGroup splits keeps one for its sink
// and residual chunks
constexpr int kShortBody = 48;

// A fixed-point grid is only formed for a maximum above this; below it the values are taken
// as zero.  For p~ this drops a tile whose probabilities are all below 1e-30 relative to the
// running maximum (whose own probability, 1, is already in l): far below fp32 resolution of
// the sums.  It keeps grid scale = bound / max finite (a denormal or tiny max would make it
// inf, and 0 * inf a NaN).
constexpr float kTinyMax = 1e-30f;

struct DecodeArgs {
    const uint8_t* k_body;
    const uint8_t* v_body;
    uint16_t* k_resid;  // written only by a fused append (step_len > 0)
    uint16_t* v_resid;
    const uint16_t* k_sink;
    const uint16_t* v_sink;
    int32_t* seq_len;   // read, and written only by a fused append
    const void* q;
    int q_bf16;
    void* out;
    int out_bf16;
    int n_kv, n_q, g, max_blocks, n_sink;
    int rotate;        // 1: body tiles hold the Hadamard-rotated domain; 0: unrotated (ablations)
    const int32_t* block_table;  // paged body: [batch][max_blocks] pool block ids, or null (dense)
    int n_phys;                  // pool size in blocks (paged)
    uint32_t* err_word;
    float scale_log2;  // sm_scale * log2(e): logits are kept in log2 units
    int n_split, bps;  // splits per stream and body tiles per body split
    int n_res;         // splits that hold only sink + residual chunks (the last n_res of n_split)
    int n_streams;     // batch * n_kv
    int n_chunk, g_chunk;  // head chunks per stream and heads per chunk (row-digit kernels)
    int group;         // > 1: the n_split splits of a stream are the waves of one workgroup
    float* ws;         // [batch][n_q][n_split][kPart] when n_split > 1
    // Fused append of a lock-step step: > 0 the common length of the sequences with the token of
    // k_new / v_new ([batch][n_kv][kD] bf16) appended as their last residual row; 0: lengths
    // from seq_len and no append.
    int step_len;
    const uint16_t* k_new;
    const uint16_t* v_new;
};

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v4f mfma_bf16(v8bf a, v8bf b, v4f c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// v_perm_b32: byte selector 0-3 picks from `lo`, 4-7 from `hi`, 0x0c gives zero.
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// The 16 codes of one unit as an int8 MFMA operand: byte q of dword s is code 4*s + q.
template <int BITS>
__device__ __forceinline__ v4i unit_i8(const uint32_t* w) {
    if constexpr (BITS == 2) {
        const uint32_t x = w[0], M = 0x03030303u;
        return v4i{(int)(x & M), (int)((x >> 2) & M), (int)((x >> 4) & M), (int)((x >> 6) & M)};
    } else {
        const uint32_t M = 0x0F0F0F0Fu;
        return v4i{(int)(w[0] & M), (int)((w[0] >> 4) & M), (int)(w[1] & M), (int)((w[1] >> 4) & M)};
    }
}

// Max in the NaN-propagating form: no operand of the reductions here is a NaN, and fmaxf would
// first quiet every operand that comes from another lane (one more instruction per step).
__device__ __forceinline__ float fmax_any(float x, float y) { return __builtin_elementwise_maximum(x, y); }

// Four values y0..y3, each a fixed-point integer plus 0x808080, to one dword per digit k whose
// byte i is the signed digit k of value i ((byte k of y_i) ^ 0x80).
__device__ __forceinline__ void digits4(uint32_t y0, uint32_t y1, uint32_t y2, uint32_t y3, uint32_t& d0,
                                        uint32_t& d1, uint32_t& d2) {
    const uint32_t t01 = perm(y1, y0, 0x05010400u), t23 = perm(y3, y2, 0x05010400u);
    d0 = perm(t23, t01, 0x05040100u) ^ 0x80808080u;
    d1 = perm(t23, t01, 0x07060302u) ^ 0x80808080u;
    const uint32_t u01 = perm(y1, y0, 0x0c0c0602u), u23 = perm(y3, y2, 0x0c0c0602u);
    d2 = perm(u23, u01, 0x05040100u) ^ 0x80808080u;
}

// Body tiles are read once per decode step: non-temporal 16-byte loads stream them from HBM
// faster than ordinary loads and leave the caches to reused data.
__device__ __forceinline__ uint4 load_stream(const uint8_t* p) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p)));
}

// Body tile addressing.  Dense bodies: tile blk of a stream at stream * max_blocks + blk.
// Paged bodies: tile kvh of pool block block_table[b][blk].  block_id_t gives the block index
// (dense) or the pool block id (paged) of the stream's body tile blk.
template <int PG>
__device__ __forceinline__ int block_id_t(const DecodeArgs& a, int b, int blk) {
    if constexpr (PG) return a.block_table[(size_t)b * a.max_blocks + blk];
    else return blk;
}
// Paged bodies: the wave checks the pool ids of its tiles [blk0, blk1) once; an id outside the
// pool sets bit 1 of err_word and the caller skips the body (nothing outside the pool is read).
__device__ __forceinline__ bool body_ids_ok(const DecodeArgs& a, int b, int blk0, int blk1, int l) {
    if (!a.block_table) return true;
    bool bad = false;
    for (int i = blk0 + l; i < blk1; i += 64) {
        const int id = a.block_table[(size_t)b * a.max_blocks + i];
        bad |= id < 0 || id >= a.n_phys;
    }
    if (!__any(bad)) return true;
    if (l == 0 && a.err_word) __hip_atomic_fetch_or(a.err_word, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return false;
}

// The aux of one K tile and one V tile as loaded for the row-digit kernels: lane l holds entries
// 2l and 2l + 1 of each row (a, b, s2 of the K tile's channels, of the V tile's tokens).  fp32:
// three 8-byte loads per tile; compact: the two binary16 offsets (4 bytes) and the two E4M3
// values of each scale row (2 bytes each).
template <int CMP>
struct HalfAux {
    uint2 a, b, s;
};
template <>
struct HalfAux<1> {
    uint32_t b, a, s;
};
__device__ __forceinline__ uint2 load_stream2(const uint8_t* p) {
    return __builtin_bit_cast(uint2, __builtin_nontemporal_load(reinterpret_cast<const v2u*>(p)));
}
template <int CMP>
__device__ __forceinline__ void load_half_aux(HalfAux<CMP>& r, const uint8_t* t, size_t cb, int l) {
    // (lane offsets as unsigned 32-bit values: the loads then take the uniform tile address as
    // their scalar base, with no 64-bit address arithmetic per lane)
    const uint8_t* x = t + cb;
    const uint32_t u = (uint32_t)l;
    if constexpr (CMP) {
        r.b = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(x + 4u * u));
        r.a = __builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(x + (256u + 2u * u)));
        r.s = __builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(x + (384u + 2u * u)));
    } else {
        r.a = load_stream2(x + 8u * u);
        r.b = load_stream2(x + (512u + 8u * u));
        r.s = load_stream2(x + (1024u + 8u * u));
    }
}
// -> fp32 rows a, b, s2 (rows r0, r0 + 1, r0 + 2 of aux), entries 2l and 2l + 1; both compact
// conversions are exact
template <int CMP>
__device__ __forceinline__ void stage_half_aux(float (&aux)[6][kD], int r0, const HalfAux<CMP>& r, int l) {
    float a0, a1, b0, b1, s0, s1;
    if constexpr (CMP) {
        const auto ap = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.a, false);
        const auto sp = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.s, false);
        a0 = ap[0];
        a1 = ap[1];
        s0 = sp[0];
        s1 = sp[1];
        b0 = (float)__builtin_bit_cast(_Float16, (uint16_t)(r.b & 0xFFFFu));
        b1 = (float)__builtin_bit_cast(_Float16, (uint16_t)(r.b >> 16));
    } else {
        a0 = __uint_as_float(r.a.x);
        a1 = __uint_as_float(r.a.y);
        b0 = __uint_as_float(r.b.x);
        b1 = __uint_as_float(r.b.y);
        s0 = __uint_as_float(r.s.x);
        s1 = __uint_as_float(r.s.y);
    }
    *reinterpret_cast<float2*>(&aux[r0][2 * l]) = make_float2(a0, a1);
    *reinterpret_cast<float2*>(&aux[r0 + 1][2 * l]) = make_float2(b0, b1);
    *reinterpret_cast<float2*>(&aux[r0 + 2][2 * l]) = make_float2(s0, s1);
}

// Orders this wave's accesses to its own LDS: a wave's LDS operations execute in issue order,
// so no wait is needed, only a point that the compiler does not move memory operations across.
// (Each wave of a decode workgroup has an LDS block of its own.)
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// LDS butterflies (stride 1..64) over rows [0, g) of x; one wave.  Unnormalized.
template <int GQ>
__device__ __forceinline__ void lds_hadamard(float (&x)[GQ][kD], int g) {
    const int l = threadIdx.x & 63;
    for (int h = 1; h < kD; h <<= 1) {
        for (int idx = l; idx < g * 64; idx += 64) {
            const int j = idx >> 6, r = idx & 63;
            const int i0 = (r / h) * 2 * h + (r % h);
            const float x0 = x[j][i0], x1 = x[j][i0 + h];
            x[j][i0] = x0 + x1;
            x[j][i0 + h] = x0 - x1;
        }
        wave_sync();
    }
}

// Query rows qrow .. qrow + g - 1 into LDS rows 0 .. NR - 1 (rows >= g zero): lane l writes
// channels 2l, 2l + 1 of every row.  One branch on the dtype, so every load is in flight before
// the first is used (q is only 4-byte aligned).
template <int NR>
__device__ __forceinline__ void q_to_lds(float (&q)[NR][kD], const DecodeArgs& a, size_t qrow, int g, int l) {
    float v0[NR], v1[NR];
    if (a.q_bf16) {
        const uint32_t* q2 = static_cast<const uint32_t*>(a.q);
#pragma unroll
        for (int h = 0; h < NR; ++h) {
            const uint32_t w = q2[(qrow + min(h, g - 1)) * (kD / 2) + l];
            v0[h] = __uint_as_float(w << 16);
            v1[h] = __uint_as_float(w & 0xFFFF0000u);
        }
    } else {
        const float* q1 = static_cast<const float*>(a.q);
#pragma unroll
        for (int h = 0; h < NR; ++h) {
            const size_t i = (qrow + min(h, g - 1)) * kD + 2 * l;
            v0[h] = q1[i];
            v1[h] = q1[i + 1];
        }
    }
#pragma unroll
    for (int h = 0; h < NR; ++h) {
        q[h][2 * l] = h < g ? v0[h] : 0.f;
        q[h][2 * l + 1] = h < g ? v1[h] : 0.f;
    }
}

// NB runs of 8 consecutive query values, run r starting at element idx[r] (a multiple of 8), with
// one branch on the dtype.
template <int NB>
__device__ __forceinline__ void load_q_runs(const DecodeArgs& a, const size_t (&idx)[NB], float (&v)[NB][8]) {
    if (a.q_bf16) {
        const uint32_t* q2 = static_cast<const uint32_t*>(a.q);
#pragma unroll
        for (int r = 0; r < NB; ++r)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t w = q2[idx[r] / 2 + e];
                v[r][2 * e] = __uint_as_float(w << 16);
                v[r][2 * e + 1] = __uint_as_float(w & 0xFFFF0000u);
            }
    } else {
        const float* q1 = static_cast<const float*>(a.q);
#pragma unroll
        for (int r = 0; r < NB; ++r)
#pragma unroll
            for (int e = 0; e < 8; ++e) v[r][e] = q1[idx[r] + e];
    }
}

// ---- group size <= 4: digit planes in the MFMA rows ----------------------------------------
// Both products take the real-valued side (q~ or p~, as base-256 digit planes) as the A operand
// and the codes as B.  Row 4*h + j of A is digit j of head h (j = 3 is zero).  The A and B
// register layouts of the 16x16x64 product are mirror images, so the code operands are the same
// registers as with codes in A.  Output lane (G, n) then receives, in its four accumulator
// registers, the digit partial sums of head G for column n (a token in QK, a channel in PV) and
// recombines them in-lane with two shifted adds.  One MFMA serves all three digits, and each
// lane finishes exactly one useful value per product.
//
// Between the products the probabilities move from the QK output layout (lane (G, n) = head G,
// token n of each 16) to the PV A layout (lane (G, 4h + j) = digit j of head h, tokens 4G..4G+3
// of each 16): a byte transpose inside each quad, then one lane permutation (ds_bpermute).

__device__ __forceinline__ int dpp_x1(int v) { return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true); }
__device__ __forceinline__ int dpp_x2(int v) { return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true); }
__device__ __forceinline__ int dpp_half_mirror(int v) { return __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true); }
__device__ __forceinline__ int dpp_mirror(int v) { return __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true); }
__device__ __forceinline__ float fdpp_x1(float v) { return __int_as_float(dpp_x1(__float_as_int(v))); }
__device__ __forceinline__ float fdpp_x2(float v) { return __int_as_float(dpp_x2(__float_as_int(v))); }
__device__ __forceinline__ float fdpp_half_mirror(float v) { return __int_as_float(dpp_half_mirror(__float_as_int(v))); }
__device__ __forceinline__ float fdpp_mirror(float v) { return __int_as_float(dpp_mirror(__float_as_int(v))); }
// max / sum over the 16 lanes of a row (lanes 16G .. 16G + 15): the quad (partners ^1, ^2), then
// the other quad of the half (mirror within 8), then the other half (mirror within 16).  Every
// step combines two equal-shaped partial results, so all 16 lanes end with identical values.
__device__ __forceinline__ float row_max(float v) {
    v = fmax_any(v, fdpp_x1(v));
    v = fmax_any(v, fdpp_x2(v));
    v = fmax_any(v, fdpp_half_mirror(v));
    return fmax_any(v, fdpp_mirror(v));
}
// The same for values >= 0: their bit patterns order as signed integers, so the steps run as
// integer max instructions with the lane move folded in.
__device__ __forceinline__ float row_max_nonneg(float v) {
    int b = __float_as_int(v);
    b = max(b, dpp_x1(b));
    b = max(b, dpp_x2(b));
    b = max(b, dpp_half_mirror(b));
    return __int_as_float(max(b, dpp_mirror(b)));
}
__device__ __forceinline__ float row_sum(float v) {
    v += fdpp_x1(v);
    v += fdpp_x2(v);
    v += fdpp_half_mirror(v);
    return v + fdpp_mirror(v);
}

// The digit-weighted sum of one output lane: register i holds the partial sum of digit i.  The
// true sum fits int32, so the wrapping arithmetic below is exact.  Horner form, two
// shift-and-add instructions (v_lshl_add_u32); the empty asm statement keeps the compiler from
// distributing the outer shift over the inner sum, which costs a third instruction.
__device__ __forceinline__ int digit_sum(v4i c) {
    uint32_t t = ((uint32_t)c[2] << 8) + (uint32_t)c[1];
    asm("" : "+v"(t));
    return (int)((t << 8) + (uint32_t)c[0]);
}

// Lane j of a quad holds y (row j of a 4 x 4 byte matrix); returns column j: byte i of the
// result is byte j of lane i's y.  Two exchanges (partners j ^ 2, then j ^ 1), each a DPP move
// and a byte permute.
__device__ __forceinline__ uint32_t quad_transpose_bytes(uint32_t y, int j) {
    const uint32_t selA = j < 2 ? 0x05040100u : 0x03020706u;
    const uint32_t selB = (j & 1) ? 0x03070105u : 0x06020400u;
    const uint32_t t = perm((uint32_t)dpp_x2((int)y), y, selA);
    return perm((uint32_t)dpp_x1((int)t), t, selB);
}

// The codes of one unit as the B operand of the row-digit kernel.  At 2 bits one shift gives
// all four byte planes: dwords 0 and 2 carry the codes, dwords 1 and 3 four times the codes;
// the A operand compensates with elements kPlaneMul times larger in dwords 0 and 2.
template <int BITS>
__device__ __forceinline__ v4i unit_planes(const uint32_t* w) {
    if constexpr (BITS == 2) {
        const uint32_t x = w[0], x4 = x >> 4, M = 0x03030303u;
        return v4i{(int)(x & M), (int)(x & (M << 2)), (int)(x4 & M), (int)(x4 & (M << 2))};
    } else {
        return unit_i8<BITS>(w);
    }
}
template <int BITS>
constexpr float kPlaneMul = BITS == 2 ? 4.f : 1.f;

// Query heads are taken in groups of four (NH groups, g <= 4 * NH): every group repeats the
// per-head work on the same code operands, which are extracted once per tile.
template <int NH, int X1>
struct Smem4 {
    float q[4 * NH + X1][kD];       // rotated q (rows >= g zero); reused for the inverse rotation of the output
    float aux[6][kD];               // a_K b_K s2_K a_V b_V s2_V of the current tile
    uint4 qp[NH][4][2][16];         // q~ digit planes [group][digit slot][kappa][qslot(slot, G, head)]; slot 3 stays zero
    uint4 qp4[X1 ? 4 : 1][2][4];    // X1: the extra head's q~ digit planes [digit slot][kappa][G]; slot 3 zero
    float hv[4 * NH + X1][4];       // per head: beta, q~ step, alpha, l
    float p[4 * NH + X1][kRC];      // probabilities of a bf16 chunk (sink / residual)
};

// Position of the 16-byte piece (K group G, head h) in a digit slot's row of the q~ planes.  The
// QK operand read has lane (G, 4h + j) fetch piece (G, h) of slot j; the slot-dependent swizzle
// gives the 16 lanes of a row 16 different bank groups (unswizzled, the four slots of one (G, h)
// share a bank group).
__device__ __forceinline__ int qslot(int slot, int G, int h) { return (4 * G + h) ^ (4 * slot); }

// Max and sum over the whole wave (the four DPP rows, then row pairs): every lane ends with
// the same value.
template <class F>
__device__ __forceinline__ float across_rows4(float v, F f) {
    const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = f(__uint_as_float(x[0]), __uint_as_float(x[1]));
    const auto y = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return f(__uint_as_float(y[0]), __uint_as_float(y[1]));
}
__device__ __forceinline__ float wave_max(float v) {
    return across_rows4(row_max(v), [](float x, float y) { return fmax_any(x, y); });
}
__device__ __forceinline__ float wave_max_nonneg(float v) {
    return across_rows4(row_max_nonneg(v), [](float x, float y) {
        return __int_as_float(max(__float_as_int(x), __float_as_int(y)));
    });
}
__device__ __forceinline__ float wave_sum(float v) {
    return across_rows4(row_sum(v), [](float x, float y) { return x + y; });
}

// Digit-weighted sum over the four row groups of a wave (lanes n, 16 + n, 32 + n, 48 + n),
// scattered: row group G receives the sum over r of x_G(row group r) * 256^r.
// permlane32_swap(a, b) returns {a's rows 0-1, b's rows 0-1} and {a's rows 2-3, b's rows 2-3}, so
// after the first two swaps a lane of row group R holds x(R mod 2) and x(R mod 2 + 2) of x0, x1
// (rows 0-1) or x2, x3 (rows 2-3); their weights differ by 256^2, so the lane adds the second
// times 2^16 and keeps the common factor 256^(R mod 2) for later.  permlane16_swap(a, b) returns
// {a's even rows in even rows, b's even rows in odd rows} and {a's odd rows in even rows, b's odd
// rows in odd rows}: the even-row partial (factor 1) plus 2^8 times the odd-row partial (factor
// 256) completes each row group's sum.  Integer arithmetic wraps exactly.
__device__ __forceinline__ uint32_t rows_digit_reduce_scatter4(uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3) {
    const auto a = __builtin_amdgcn_permlane32_swap(x0, x2, false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(x1, x3, false, false);
    const auto c = __builtin_amdgcn_permlane16_swap(a[0] + (a[1] << 16), b[0] + (b[1] << 16), false, false);
    return c[0] + (c[1] << 8);
}

// X1 = 1 (group size 5, with NH = 1): a fifth query head spread over the whole wave instead of a
// second head group of four slots, carried by the head group's own products in the digit slot
// the group leaves empty: q~ and p~ have three digits, so A row 4 h + 3 (slot 3 of head h) is
// zero, and rows 3, 7 and 11 take the extra head's digits 0, 1 and 2.  Accumulator 3 of lane
// (G, n) then holds its digit-G partial sum for column n (a token in QK, a channel in PV; row
// group 3 gets zero from row 15), and a reduce-scatter over the row groups combines the digits
// so that lane (G, n) holds the head's logits for tokens 64 sg + 16 G + n and its outputs for
// channels 16 (4 q + G) + n (sg, q = 0, 1): two values per lane, no padded head slots and no
// MFMA of its own.
template <int BITS, int NH, int CMP, int PG, int X1>
__global__ __launch_bounds__(64 * kMaxGroup) __attribute__((amdgpu_waves_per_eu(BITS == 2 && NH == 1 && !X1 ? 3 : 2, 8)))
void k_decode4(DecodeArgs a) {
    static_assert(X1 == 0 || NH == 1, "the extra head is only for one head group");
    // one LDS block per wave (dynamic: one to kMaxGroup waves per workgroup)
    extern __shared__ __align__(16) unsigned char dyn_lds[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    Smem4<NH, X1>& sm = reinterpret_cast<Smem4<NH, X1>*>(dyn_lds)[wave];
    constexpr int WPU = BITS / 2;
    constexpr int NHD = 4 * NH;   // head slots of the head groups
    constexpr int NHX = NHD + X1;  // all head slots
    // Fixed point: q~ and p~ in even dwords of the A operand are scaled by MUL (the code planes
    // there are not shifted up), so every product term carries weight MUL.  The exact sum is
    // bounded by MUL * (2^BITS - 1) * 128 * QMAX < 2^31 and MUL * QMAX < 2^22 keeps the
    // rounding below exact.
    constexpr float MUL = kPlaneMul<BITS>;
    constexpr int QMAX = 1048575;
    constexpr float MAGIC = 12582912.f;  // 1.5 * 2^23: x + MAGIC rounds x to an integer
    constexpr uint32_t MAGIC_BITS = 0x4B400000u;
    // output role: head 4*hg + G, column n; A-operand role: row 4*h + j (digit j of head 4*hg + h)
    const int l = threadIdx.x & 63, G = l >> 4, n = l & 15, h = (l >> 2) & 3, j = l & 3;
    // wave = (head chunk, stream, split), the chunk slowest: the chunks of a stream read the
    // same tiles, n_streams * n_split waves apart, which keeps them on one XCD when that
    // distance in workgroups is a multiple of 8.  In group mode a workgroup's waves are the
    // stream's splits.
    const int split = a.group > 1 ? wave : blockIdx.x % a.n_split;
    const int cs = a.group > 1 ? blockIdx.x : blockIdx.x / a.n_split;
    const int stream = cs % a.n_streams, chunk = cs / a.n_streams;
    const int g = min(a.g_chunk, a.g - chunk * a.g_chunk);  // query heads of this wave
    const int b = stream / a.n_kv, kvh = stream % a.n_kv;
    // A fused append takes the step's length from the host.  The stored length must then be the
    // one before the append, or the one after it (kv head 0 stores it, perhaps already); else the
    // sequence is left as it is and bit 2 of err_word is set.
    const int stored = a.seq_len[b];
    const bool step_ok = a.step_len == 0 || stored == a.step_len - 1 || stored == a.step_len;
    const int len = a.step_len > 0 ? a.step_len : max(stored, 0);
    const int ns = min(len, a.n_sink);
    const int nbody = min(len > a.n_sink ? (len - a.n_sink) / kG : 0, a.max_blocks);
    const int nr = len > a.n_sink ? (len - a.n_sink) % kG : 0;
    // The last n_res splits hold only sink + residual chunks; without them the body splits share
    // those chunks.
    const int nbs = a.n_split - a.n_res;  // body splits
    const bool res_only = split >= nbs;
    const bool body_last = split == nbs - 1;  // takes any excess of body tiles
    const int blk0 = res_only ? 0 : split * a.bps;
    int blk1 = res_only ? 0 : (body_last ? nbody : min(blk0 + a.bps, nbody));
    if (PG && blk0 < blk1 && !body_ids_ok(a, b, blk0, blk1, l)) blk1 = blk0;
    const size_t qrow = (size_t)b * a.n_q + (size_t)kvh * a.g + (size_t)chunk * a.g_chunk;
    const size_t tb = tile_bytes(BITS, CMP), cb = code_bytes(BITS);

    float m_run[NH], l_run[NH];  // head 4*hg + G; l_run is this lane's partial sum
    float orot[NH][8];           // head 4*hg + G, channel 16*mt + n (rotated domain)
    // X1: the extra head's running max, this lane's partial sum, and its output channels
    // 16 (4 q + G) + n, q = 0, 1
    float m4 = -INFINITY, l4 = 0.f, orot4[2] = {0.f, 0.f};
#pragma unroll
    for (int hg = 0; hg < NH; ++hg) {
        m_run[hg] = -INFINITY;
        l_run[hg] = 0.f;
#pragma unroll
        for (int mt = 0; mt < 8; ++mt) orot[hg][mt] = 0.f;
    }

    // online softmax of group hg over this lane's logits (log2 units; -inf = absent) -> p,
    // returns alpha
    auto softmax_update = [](auto& lg, bool maybe_absent, float& m, float& lsum) -> float {
        constexpr int N = sizeof(lg) / sizeof(lg[0]);
        float mx = lg[0];
#pragma unroll
        for (int k = 1; k < N; ++k) mx = fmaxf(mx, lg[k]);
        mx = row_max(mx);
        const float m_new = fmaxf(m, mx);
        const float alpha = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - m_new);
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < N; ++k) {
            float p = __builtin_amdgcn_exp2f(lg[k] - m_new);
            if (maybe_absent) p = lg[k] == -INFINITY ? 0.f : p;
            lg[k] = p;
            s += p;
        }
        lsum = lsum * alpha + s;
        m = m_new;
        return alpha;
    };

    // the same for the extra head, whose 128 logits are spread over the wave (two per lane)
    auto softmax_wave = [](float (&lg)[2], bool maybe_absent, float& m, float& lsum) -> float {
        const float mx = wave_max(fmaxf(lg[0], lg[1]));
        const float m_new = fmaxf(m, mx);
        const float alpha = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - m_new);
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            float p = __builtin_amdgcn_exp2f(lg[k] - m_new);
            if (maybe_absent) p = lg[k] == -INFINITY ? 0.f : p;
            lg[k] = p;
            s += p;
        }
        lsum = lsum * alpha + s;
        m = m_new;
        return alpha;
    };

    if (blk0 < blk1) {
        // Two register buffers, one tile each, alternate between tiles.  While a tile is
        // consumed from one, the next tile's parts go into the other: its aux right after the
        // current aux is staged in LDS, its key codes after the QK products, its value codes
        // after the PV products.  The first tile's loads go out before the query set-up.  No
        // load sits behind a branch (the prefetch past the last tile re-reads that tile), so
        // each wait counts exactly the loads it needs.
        struct TileRegs {
            uint4 k[2][2 * WPU], v[2][2 * WPU];
            HalfAux<CMP> ak, av;
        };
        TileRegs ra, rb;
        // tiles by block_id (pool id when paged); the id of the next tile is read a tile ahead
        auto tile_of = [&](int id) { return PG ? (size_t)id * a.n_kv + kvh : (size_t)stream * a.max_blocks + id; };
        auto tile_k = [&](int id) { return a.k_body + tile_of(id) * tb; };
        auto tile_v = [&](int id) { return a.v_body + tile_of(id) * tb; };
        auto load_aux = [&](TileRegs& r, int id) {
            load_half_aux<CMP>(r.ak, tile_k(id), cb, l);
            load_half_aux<CMP>(r.av, tile_v(id), cb, l);
        };
        auto load_codes = [&](const uint8_t* t, uint4 (&c)[2][2 * WPU]) {
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int k = 0; k < 2 * WPU; ++k) c[s][k] = load_stream(t + 16u * (unsigned)(s * 128 * WPU + 64 * k + l));
        };
        const int id0 = block_id_t<PG>(a, b, blk0);
        load_codes(tile_k(id0), ra.k);
        load_codes(tile_v(id0), ra.v);
        load_aux(ra, id0);

        q_to_lds<NHX>(sm.q, a, qrow, g, l);
        for (int idx = l; idx < NH * 32; idx += 64)
            sm.qp[idx >> 5][3][(idx >> 4) & 1][idx & 15] = make_uint4(0u, 0u, 0u, 0u);
        if (X1 && l < 8) sm.qp4[X1 ? 3 : 0][l >> 2][l & 3] = make_uint4(0u, 0u, 0u, 0u);
        wave_sync();
        if (a.rotate) lds_hadamard<NHX>(sm.q, g);
        // q~ role: head 4*hg + G, channels 8n .. 8n + 7 (rotated and normalized, or as given)
        const float qs = a.rotate ? kInvSqrt128 : 1.f;
        // two head groups: q stays in LDS (each lane scales, and later reads, only its own
        // elements), which keeps 16 registers free for the tile loop
        constexpr bool QLDS = NH == 2;
        float qr[QLDS ? 1 : NH][8];
#pragma unroll
        for (int hg = 0; hg < NH; ++hg)
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                if constexpr (QLDS) sm.q[4 * hg + G][8 * n + k] *= qs;
                else qr[hg][k] = sm.q[4 * hg + G][8 * n + k] * qs;
            }
        // extra head: channels 2l, 2l + 1
        const float qr4[2] = {X1 ? sm.q[NHX - 1][2 * l] * qs : 0.f, X1 ? sm.q[NHX - 1][2 * l + 1] * qs : 0.f};
        // source lane of the PV operand permutation (see above), as a byte address; for the
        // extra head the source row is the token block (tau), not the head
        const int perm_addr = (16 * h + 4 * G + j) * 4;
        // extra head: A row 4 h + 3 (h < 3) takes digit h from lane 4 G + h of token block tau
        const bool x1_row = X1 && j == 3 && h < 3;
        const int perm4 = (4 * G + h) * 4;

        // One tile: consume cur, prefetch tile id_next into nxt.
        // zoff is 0; the odd last tile passes it through an empty asm statement, so that its LDS
        // offsets are formed after the loop rather than held in registers across it (which spilled
        // them in the largest variant)
        auto step = [&](TileRegs& cur, TileRegs& nxt, int id_next, int zoff) {
            wave_sync();  // the previous tile is done with sm.aux / sm.qp / sm.hv
            // aux rows a_K, b_K, s2_K (keys: per channel), a_V, b_V, s2_V (values: per token)
            stage_half_aux<CMP>(sm.aux, 0, cur.ak, l);
            stage_half_aux<CMP>(sm.aux, 3, cur.av, l);
            load_aux(nxt, id_next);
            wave_sync();
            uint32_t kw[2][8 * WPU], vw[2][8 * WPU];
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int k = 0; k < 2 * WPU; ++k) {
                    kw[s][4 * k] = cur.k[s][k].x; kw[s][4 * k + 1] = cur.k[s][k].y;
                    kw[s][4 * k + 2] = cur.k[s][k].z; kw[s][4 * k + 3] = cur.k[s][k].w;
                    vw[s][4 * k] = cur.v[s][k].x; vw[s][4 * k + 1] = cur.v[s][k].y;
                    vw[s][4 * k + 2] = cur.v[s][k].z; vw[s][4 * k + 3] = cur.v[s][k].w;
                }
            // q~ = q_rot * a_K as fixed point on a per-head grid, then three digit planes; beta =
            // sum over channels of q_rot * b_K, the offsets' part of the logit (unscaled)
            {
                const float4 a0 = *reinterpret_cast<const float4*>(&sm.aux[0][8 * n]);
                const float4 a1 = *reinterpret_cast<const float4*>(&sm.aux[0][8 * n + 4]);
                const float4 b0 = *reinterpret_cast<const float4*>(&sm.aux[1][8 * n]);
                const float4 b1 = *reinterpret_cast<const float4*>(&sm.aux[1][8 * n + 4]);
                const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
                const float bk[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
                // channels 8n .. 8n + 7 = kappa n / 8, group (n % 8) / 2, components 2 (n % 2) + {0, 1}
                const int kap = n >> 3, Gq = (n >> 1) & 3, half = n & 1;
#pragma unroll
                for (int hg = 0; hg < NH; ++hg) {
                    float qv[8], qt[8], mx = 0.f;
                    if constexpr (QLDS) {
                        const float4 x0 = *reinterpret_cast<const float4*>(&sm.q[4 * hg + G][8 * n]);
                        const float4 x1 = *reinterpret_cast<const float4*>(&sm.q[4 * hg + G][8 * n + 4]);
                        qv[0] = x0.x; qv[1] = x0.y; qv[2] = x0.z; qv[3] = x0.w;
                        qv[4] = x1.x; qv[5] = x1.y; qv[6] = x1.z; qv[7] = x1.w;
                    } else {
#pragma unroll
                        for (int k = 0; k < 8; ++k) qv[k] = qr[QLDS ? 0 : hg][k];
                    }
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        qt[k] = qv[k] * av[k];
                        mx = fmaxf(mx, fabsf(qt[k]));
                    }
                    mx = row_max_nonneg(mx);
                    const float sc = mx > kTinyMax ? (float)QMAX * __builtin_amdgcn_rcpf(mx) : 0.f;
                    // channels 8n .. 8n + 3 sit in an even dword of the A operand, 8n + 4 ..
                    // 8n + 7 in an odd one
                    float bsum = 0.f;
                    uint32_t y[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const float yf = fmaf(qt[k], k < 4 ? sc * MUL : sc, MAGIC);
                        bsum = fmaf(qv[k], bk[k], bsum);
                        y[k] = __float_as_uint(yf) + (0x808080u - MAGIC_BITS);
                    }
                    const float bs = row_sum(bsum);
                    uint32_t d0, d1, d2, e0, e1, e2;
                    digits4(y[0], y[1], y[2], y[3], d0, d1, d2);
                    digits4(y[4], y[5], y[6], y[7], e0, e1, e2);
                    reinterpret_cast<uint2*>(&sm.qp[hg][0][kap][qslot(0, Gq, G)])[half] = make_uint2(d0, e0);
                    reinterpret_cast<uint2*>(&sm.qp[hg][1][kap][qslot(1, Gq, G)])[half] = make_uint2(d1, e1);
                    reinterpret_cast<uint2*>(&sm.qp[hg][2][kap][qslot(2, Gq, G)])[half] = make_uint2(d2, e2);
                    if (n == 0) {
                        sm.hv[4 * hg + G][0] = bs;
                        sm.hv[4 * hg + G][1] = mx * (1.0f / (MUL * (float)QMAX));
                    }
                }
                if constexpr (X1) {
                    // extra head: channels 2l, 2l + 1 = kappa l / 32, group (l / 8) % 4, bytes
                    // 2 (l % 8) + {0, 1} of that group (an even dword when (l / 2) % 2 == 0);
                    // grid, digits and beta as for the head groups, over the whole wave
                    const float2 a2 = *reinterpret_cast<const float2*>(&sm.aux[0][2 * l]);
                    const float2 b2 = *reinterpret_cast<const float2*>(&sm.aux[1][2 * l]);
                    const float qt0 = qr4[0] * a2.x, qt1 = qr4[1] * a2.y;
                    const float mx = wave_max_nonneg(fmaxf(fabsf(qt0), fabsf(qt1)));
                    const float sc = mx > kTinyMax ? (float)QMAX * __builtin_amdgcn_rcpf(mx) : 0.f;
                    const bool even = ((l >> 1) & 1) == 0;
                    const float y0f = fmaf(qt0, even ? sc * MUL : sc, MAGIC);
                    const float y1f = fmaf(qt1, even ? sc * MUL : sc, MAGIC);
                    const float bs = wave_sum(fmaf(qr4[1], b2.y, qr4[0] * b2.x));
                    const uint32_t y0 = __float_as_uint(y0f) + (0x808080u - MAGIC_BITS);
                    const uint32_t y1 = __float_as_uint(y1f) + (0x808080u - MAGIC_BITS);
                    const uint32_t d01 = perm(y1, y0, 0x05010400u) ^ 0x80808080u;  // digit 0 | digit 1 pairs
                    const uint32_t d2 = perm(y1, y0, 0x0c0c0602u) ^ 0x8080u;       // digit 2 pair
                    const int kp = l >> 5, gq = (l >> 3) & 3, e = l & 7;
                    reinterpret_cast<uint16_t*>(&sm.qp4[0][kp][gq])[e] = (uint16_t)(d01 & 0xFFFFu);
                    reinterpret_cast<uint16_t*>(&sm.qp4[X1 ? 1 : 0][kp][gq])[e] = (uint16_t)(d01 >> 16);
                    reinterpret_cast<uint16_t*>(&sm.qp4[X1 ? 2 : 0][kp][gq])[e] = (uint16_t)d2;
                    if (l == 0) {
                        sm.hv[NHX - 1][0] = bs;
                        sm.hv[NHX - 1][1] = mx * (1.0f / (MUL * (float)QMAX));
                    }
                }
            }
            wave_sync();

            // logits of head 4*hg + G, token 64*sg + 16*tau + n.  Tokens outer, head groups
            // inner: the code planes of a token block are extracted once and used at once.
            float lg[NH][8];
            v4i aq[NH][2];
            float bq[NH], fqs[NH];  // beta and the q~ grid step in logit units (log2, scaled)
#pragma unroll
            for (int hg = 0; hg < NH; ++hg) {
#pragma unroll
                for (int kap = 0; kap < 2; ++kap) {
                    // X1: rows 3, 7, 11 (slot 3 of heads 0-2) take the extra head's digits 0-2
                    const int jq = j + zoff;
                    const uint4 u = X1 && j == 3 && h < 3 ? sm.qp4[X1 ? h : 0][kap][G] : sm.qp[hg][jq][kap][qslot(jq, G, h)];
                    aq[hg][kap] = v4i{(int)u.x, (int)u.y, (int)u.z, (int)u.w};
                }
                fqs[hg] = sm.hv[4 * hg + G][1] * a.scale_log2;
                bq[hg] = sm.hv[4 * hg + G][0] * a.scale_log2;
            }
            // X1: accumulator 3 holds the extra head's digit-G partial (row group 3: zero)
            uint32_t x4[2][4];
#pragma unroll
            for (int sg = 0; sg < 2; ++sg)
#pragma unroll
                for (int tau = 0; tau < 4; ++tau) {
                    const v4i b0 = unit_planes<BITS>(&kw[sg][(2 * tau) * WPU]);
                    const v4i b1 = unit_planes<BITS>(&kw[sg][(2 * tau + 1) * WPU]);
                    const float s2k = sm.aux[2][64 * sg + 16 * tau + n];
#pragma unroll
                    for (int hg = 0; hg < NH; ++hg) {
                        v4i c = mfma_i8(aq[hg][0], b0, v4i{0, 0, 0, 0});
                        c = mfma_i8(aq[hg][1], b1, c);
                        lg[hg][4 * sg + tau] = fmaf((float)digit_sum(c), fqs[hg], bq[hg]) * s2k;
                        if (X1 && hg == 0) x4[sg][tau] = (uint32_t)c[3];
                    }
                }
            float lg4[2] = {0.f, 0.f};  // extra head, tokens 64 sg + 16 G + n
            if constexpr (X1) {
                const float fqs4 = sm.hv[NHX - 1][1] * a.scale_log2, bq4 = sm.hv[NHX - 1][0] * a.scale_log2;
#pragma unroll
                for (int sg = 0; sg < 2; ++sg) {
                    const uint32_t raw = rows_digit_reduce_scatter4(x4[sg][0], x4[sg][1], x4[sg][2], x4[sg][3]);
                    lg4[sg] = fmaf((float)(int)raw, fqs4, bq4) * sm.aux[2][64 * sg + 16 * G + n];
                }
            }
            load_codes(tile_k(id_next), nxt.k);

            // extra head: lane (G, n) holds token 64 sg + 16 G + n, i.e. token block tau = G of
            // each sg; its digit words are byte-transposed like the head groups' and reach A rows
            // 3, 7, 11 (digit h in row 4 h + 3) from the lanes of token block tau
            float alpha4 = 0.f, gam4 = 0.f, fp4 = 0.f;
            uint32_t t4[2] = {0u, 0u};
            if constexpr (X1) {
                alpha4 = softmax_wave(lg4, false, m4, l4);
                // the offsets' part of the output: sum over tokens of p * b_V
                gam4 = wave_sum(fmaf(lg4[1], sm.aux[4][64 + 16 * G + n], lg4[0] * sm.aux[4][16 * G + n]));
                lg4[0] *= sm.aux[3][16 * G + n];
                lg4[1] *= sm.aux[3][64 + 16 * G + n];
                const float pmx = wave_max_nonneg(fmaxf(lg4[0], lg4[1]));
                const float psc = pmx > kTinyMax ? (float)QMAX * __builtin_amdgcn_rcpf(pmx) : 0.f;
                const float ps = (G & 1) ? psc : psc * MUL;
#pragma unroll
                for (int sg = 0; sg < 2; ++sg) {
                    const float yf = fmaf(lg4[sg], ps, MAGIC);
                    t4[sg] = quad_transpose_bytes(__float_as_uint(yf) + (0x80808080u - MAGIC_BITS), j);
                }
                fp4 = pmx * (1.0f / (MUL * (float)QMAX));
            }
            v4i ap[NH][2];
            float alpha[NH], gam[NH], fp[NH];  // gam: the offset term in output units
#pragma unroll
            for (int hg = 0; hg < NH; ++hg) {
                alpha[hg] = softmax_update(lg[hg], false, m_run[hg], l_run[hg]);
                // the offsets' part of the output, sum over tokens of p * b_V; then p * a_V, the
                // real-valued side of the code products
                float pmx = 0.f, gsum = 0.f;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int tok = 64 * (k >> 2) + 16 * (k & 3) + n;
                    gsum = fmaf(lg[hg][k], sm.aux[4][tok], gsum);
                    lg[hg][k] *= sm.aux[3][tok];
                    pmx = fmaxf(pmx, lg[hg][k]);
                }
                pmx = row_max_nonneg(pmx);
                const float psc = pmx > kTinyMax ? (float)QMAX * __builtin_amdgcn_rcpf(pmx) : 0.f;
#pragma unroll
                for (int sg = 0; sg < 2; ++sg) {
                    uint32_t D[4];
#pragma unroll
                    for (int tau = 0; tau < 4; ++tau) {
                        const float yf = fmaf(lg[hg][4 * sg + tau], (tau & 1) ? psc : psc * MUL, MAGIC);
                        const uint32_t y = __float_as_uint(yf) + (0x80808080u - MAGIC_BITS);
                        const uint32_t t = quad_transpose_bytes(y, j);
                        uint32_t d = (uint32_t)__builtin_amdgcn_ds_bpermute(perm_addr, (int)t);
                        if (X1 && hg == 0) {
                            const uint32_t d4 = (uint32_t)__builtin_amdgcn_ds_bpermute(perm4 + 64 * tau, (int)t4[sg]);
                            d = x1_row ? d4 : d;
                        }
                        D[tau] = d ^ 0x80808080u;
                    }
                    ap[hg][sg] = v4i{(int)D[0], (int)D[1], (int)D[2], (int)D[3]};
                }
                fp[hg] = pmx * (1.0f / (MUL * (float)QMAX));
                gam[hg] = row_sum(gsum);
            }
            uint32_t x5[8];  // X1: accumulator 3, the extra head's digit-G partial of channel block mt
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) {
                const v4i v0 = unit_planes<BITS>(&vw[0][mt * WPU]);
                const v4i v1 = unit_planes<BITS>(&vw[1][mt * WPU]);
                const float s2v = sm.aux[5][16 * mt + n];
#pragma unroll
                for (int hg = 0; hg < NH; ++hg) {
                    v4i acc = mfma_i8(ap[hg][0], v0, v4i{0, 0, 0, 0});
                    acc = mfma_i8(ap[hg][1], v1, acc);
                    orot[hg][mt] = fmaf(fmaf((float)digit_sum(acc), fp[hg], gam[hg]), s2v, orot[hg][mt] * alpha[hg]);
                    if (X1 && hg == 0) x5[mt] = (uint32_t)acc[3];
                }
            }
            if constexpr (X1) {
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const uint32_t raw = rows_digit_reduce_scatter4(x5[4 * q], x5[4 * q + 1], x5[4 * q + 2], x5[4 * q + 3]);
                    orot4[q] = fmaf(fmaf((float)(int)raw, fp4, gam4), sm.aux[5][16 * (4 * q + G) + n], orot4[q] * alpha4);
                }
            }
            load_codes(tile_v(id_next), nxt.v);
        };
        // Tiles in pairs, alternating the buffers, so that no register copy (and no wait for a
        // prefetch) is needed between iterations.
        int blk = blk0;
        int id_n = block_id_t<PG>(a, b, min(blk0 + 1, blk1 - 1));
        for (; blk + 1 < blk1; blk += 2) {
            const int id_nn = block_id_t<PG>(a, b, min(blk + 2, blk1 - 1));
            step(ra, rb, id_n, 0);
            id_n = block_id_t<PG>(a, b, min(blk + 3, blk1 - 1));
            step(rb, ra, id_nn, 0);
        }
        if (blk < blk1) {
            int z = 0;
            asm volatile("" : "+v"(z));
            step(ra, rb, id_n, z);
        }
    }

    // ---- sink and residual (bf16, unrotated) -------------------------------------------------
    // In chunks of kRC tokens: the sink's, then the residual's (no chunk spans both).  Split r of
    // the n_res sink/residual splits takes chunks r, r + n_res, ...; without such splits, split r
    // of the stream takes chunks r, r + n_split, ....  A chunk's key rows (bf16 MFMA operands)
    // and value rows (one dword per lane and row) are loaded together, one memory round trip per
    // chunk.
    float oplain[NHX][2];  // head hh, channel 2*l + jj (unrotated)
#pragma unroll
    for (int hh = 0; hh < NHX; ++hh) oplain[hh][0] = oplain[hh][1] = 0.f;
    const int nsc = (ns + kRC - 1) / kRC, nch = nsc + (nr + kRC - 1) / kRC;
    const int c0 = res_only ? split - nbs : split, cstep = res_only ? a.n_res : a.n_split;
    if ((res_only || a.n_res == 0) && c0 < nch) {
        // A operand of group hg: row 4h holds q of head 4*hg + h rounded to bf16, row 4h + 1 the
        // remainder (zero for bf16 q), rows 4h + 2, 4h + 3 zero; lane (G, 4h + j) holds
        // q[.][32k + 8G ..].  Loads are clamped to a valid head, then masked.
        v8bf aqs[NH][4];
        {
            size_t qi[4 * NH];
            float qv[4 * NH][8];
#pragma unroll
            for (int hg = 0; hg < NH; ++hg)
#pragma unroll
                for (int k = 0; k < 4; ++k) qi[4 * hg + k] = (qrow + min(4 * hg + h, g - 1)) * kD + 32 * k + 8 * G;
            load_q_runs<4 * NH>(a, qi, qv);
#pragma unroll
            for (int hg = 0; hg < NH; ++hg) {
                const bool use = 4 * hg + h < g && j < 2;
#pragma unroll
                for (int k = 0; k < 4; ++k)
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float v = use ? qv[4 * hg + k][e] : 0.f;
                        const __bf16 hi = (__bf16)v;
                        aqs[hg][k][e] = j == 0 ? hi : (__bf16)(v - (float)hi);
                    }
            }
        }
        // extra head: the same rows (hi, lo) of its q, placed in row group tau at use
        v8bf aqs4[4];
        if constexpr (X1) {
            size_t qi[4];
            float qv[4][8];
#pragma unroll
            // (clamped to a head of the chunk: the extra slot may be empty in a chunk of a larger
            // group, and its results are then not written)
            for (int k = 0; k < 4; ++k) qi[k] = (qrow + min(NHX - 1, g - 1)) * kD + 32 * k + 8 * G;
            load_q_runs<4>(a, qi, qv);
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float v = j < 2 ? qv[k][e] : 0.f;
                    const __bf16 hi = (__bf16)v;
                    aqs4[k][e] = j == 0 ? hi : (__bf16)(v - (float)hi);
                }
        }
        for (int c = c0; c < nch; c += cstep) {
            const bool in_sink = c < nsc;
            const int t0 = kRC * (in_sink ? c : c - nsc);
            const int cn = min(kRC, (in_sink ? ns : nr) - t0);
            const size_t row0 = in_sink ? (size_t)stream * a.n_sink + t0 : (size_t)stream * kG + t0;
            const uint16_t* Kp = (in_sink ? a.k_sink : a.k_resid) + row0 * kD;
            const uint16_t* Vp = (in_sink ? a.v_sink : a.v_resid) + row0 * kD;
            // A fused append's token is the residual's last row (of the last chunk): read from
            // the input, and stored into the residual below.
            const bool new_row = a.step_len > 0 && c == nch - 1;
            const uint16_t* Klast = new_row ? a.k_new + (size_t)stream * kD : Kp + (size_t)(cn - 1) * kD;
            const uint16_t* Vlast = new_row ? a.v_new + (size_t)stream * kD : Vp + (size_t)(cn - 1) * kD;
            // Rows past the chunk read its last row (in bounds) and are masked (p = 0).
            v8bf B[2][4];  // key rows 16 tau + n, channels 32 k + 8 G ..
#pragma unroll
            for (int tau = 0; tau < 2; ++tau) {
                const int i = 16 * tau + n;
                const uint16_t* kr = (i < cn - 1 ? Kp + (size_t)i * kD : Klast) + 8 * G;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint4 u = *reinterpret_cast<const uint4*>(kr + 32 * k);
                    __builtin_memcpy(&B[tau][k], &u, 16);
                }
            }
            uint32_t v2[kRC];  // value row t, channels 2 l, 2 l + 1
#pragma unroll
            for (int t = 0; t < kRC; ++t) v2[t] = reinterpret_cast<const uint32_t*>(t < cn - 1 ? Vp + (size_t)t * kD : Vlast)[l];
            if (new_row && chunk == 0 && step_ok) {
                // the token into the residual (one head chunk writes it), and the step's length
                // (kv head 0 of the sequence writes it)
                reinterpret_cast<uint32_t*>(a.k_resid + (row0 + cn - 1) * kD)[l] = reinterpret_cast<const uint32_t*>(Klast)[l];
                reinterpret_cast<uint32_t*>(a.v_resid + (row0 + cn - 1) * kD)[l] = reinterpret_cast<const uint32_t*>(Vlast)[l];
                if (kvh == 0 && l == 0) __hip_atomic_store(a.seq_len + b, a.step_len, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            if (new_row && chunk == 0 && !step_ok && l == 0 && a.err_word)
                __hip_atomic_fetch_or(a.err_word, 4u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            wave_sync();  // the previous chunk is done with sm.p / sm.hv
            // logits of head 4*hg + G, token 16*tau + n
            float lg[NH][2];
            v4f r4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int tau = 0; tau < 2; ++tau) {
#pragma unroll
                for (int hg = 0; hg < NH; ++hg) {
                    v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int k = 0; k < 4; ++k) acc = mfma_bf16(aqs[hg][k], B[tau][k], acc);
                    lg[hg][tau] = 16 * tau + n < cn ? (acc[0] + acc[1]) * a.scale_log2 : -INFINITY;
                }
                if constexpr (X1) {
                    // token block tau lands in lanes G == tau of the accumulator
                    const bool mine = h == tau;
                    const v8bf zb = {};
#pragma unroll
                    for (int k = 0; k < 4; ++k) r4 = mfma_bf16(mine ? aqs4[k] : zb, B[tau][k], r4);
                }
            }
            if constexpr (X1) {
                // extra head, token 16 G + n (G < 2)
                float lgx[2] = {G < 2 && 16 * G + n < cn ? (r4[0] + r4[1]) * a.scale_log2 : -INFINITY, -INFINITY};
                const float alpha = softmax_wave(lgx, true, m4, l4);
                orot4[0] *= alpha;
                orot4[1] *= alpha;
                if (G < 2) sm.p[NHX - 1][16 * G + n] = lgx[0];
                if (l == 0) sm.hv[NHX - 1][2] = alpha;
            }
#pragma unroll
            for (int hg = 0; hg < NH; ++hg) {
                const float alpha = softmax_update(lg[hg], true, m_run[hg], l_run[hg]);
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) orot[hg][mt] *= alpha;
                // every head slot writes its row (slots past g: p = 0, alpha = 1), so that the
                // PV loop below runs over all slots without a branch per head and token
                const bool real = 4 * hg + G < g;
#pragma unroll
                for (int tau = 0; tau < 2; ++tau) sm.p[4 * hg + G][16 * tau + n] = real ? lg[hg][tau] : 0.f;
                if (n == 0) sm.hv[4 * hg + G][2] = real ? alpha : 1.f;
            }
            wave_sync();
            // o_plain[h] = alpha o_plain[h] + sum over the chunk's rows of p[h][t] V[t]
#pragma unroll
            for (int hh = 0; hh < NHX; ++hh) {
                const float al = sm.hv[hh][2];
                oplain[hh][0] *= al;
                oplain[hh][1] *= al;
#pragma unroll
                for (int t = 0; t < kRC; t += 4) {
                    const float4 ph = *reinterpret_cast<const float4*>(&sm.p[hh][t]);
                    const float pv[4] = {ph.x, ph.y, ph.z, ph.w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        oplain[hh][0] = fmaf(pv[i], __uint_as_float(v2[t + i] << 16), oplain[hh][0]);
                        oplain[hh][1] = fmaf(pv[i], __uint_as_float(v2[t + i] & 0xFFFF0000u), oplain[hh][1]);
                    }
                }
            }
        }
    }

    // ---- finish ------------------------------------------------------------------------------
    float lt[NH];
#pragma unroll
    for (int hg = 0; hg < NH; ++hg) lt[hg] = row_sum(l_run[hg]);
    float lt4 = X1 ? wave_sum(l4) : 0.f;
    if (a.group > 1) {
        // Log-sum-exp of the splits inside the workgroup: every wave w > 0 leaves its part
        // (rotated output per head and channel, plain output, m and l per head slot) in its own
        // LDS block; wave 0 rescales all parts to their common maximum, adds them in wave order
        // and writes the output as an unsplit stream does.
        auto part = [&](int w) { return reinterpret_cast<float*>(reinterpret_cast<Smem4<NH, X1>*>(dyn_lds) + w); };
        // in each block: [NHX][kD] rotated output, [NHX][kD] plain output, [NHX] m, [NHX] l; block
        // 1 also [NHX] m of wave 0
        constexpr int XP = NHX * kD, XM = 2 * NHX * kD;
        static_assert(sizeof(Smem4<NH, X1>) >= sizeof(float) * (2 * NHX * kD + 3 * NHX), "exchange area");
        if (wave > 0) {
            float* xb = part(wave);
#pragma unroll
            for (int hg = 0; hg < NH; ++hg) {
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) xb[(4 * hg + G) * kD + 16 * mt + n] = orot[hg][mt];
                if (n == 0) {
                    xb[XM + 4 * hg + G] = m_run[hg];
                    xb[XM + NHX + 4 * hg + G] = lt[hg];
                }
            }
            if constexpr (X1) {
#pragma unroll
                for (int q = 0; q < 2; ++q) xb[(NHX - 1) * kD + 16 * (4 * q + G) + n] = orot4[q];
                if (l == 0) {
                    xb[XM + NHX - 1] = m4;
                    xb[XM + 2 * NHX - 1] = lt4;
                }
            }
#pragma unroll
            for (int hh = 0; hh < NHX; ++hh)
                *reinterpret_cast<float2*>(xb + XP + hh * kD + 2 * l) = make_float2(oplain[hh][0], oplain[hh][1]);
        }
        __syncthreads();
        if (wave > 0) return;
        const int np = a.group;
        auto ex = [](float m, float M) { return m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M); };
#pragma unroll
        for (int hg = 0; hg < NH; ++hg) {
            const int hs = 4 * hg + G;
            float M = m_run[hg];
            for (int w = 1; w < np; ++w) M = fmaxf(M, part(w)[XM + hs]);
            const float w0 = ex(m_run[hg], M);
            lt[hg] *= w0;
#pragma unroll
            for (int mt = 0; mt < 8; ++mt) orot[hg][mt] *= w0;
            for (int w = 1; w < np; ++w) {
                const float* xb = part(w);
                const float ww = ex(xb[XM + hs], M);
                lt[hg] = fmaf(ww, xb[XM + NHX + hs], lt[hg]);
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) orot[hg][mt] = fmaf(ww, xb[hs * kD + 16 * mt + n], orot[hg][mt]);
            }
            if (n == 0) part(1)[XM + 2 * NHX + hs] = m_run[hg];
        }
        if constexpr (X1) {
            float M = m4;
            for (int w = 1; w < np; ++w) M = fmaxf(M, part(w)[XM + NHX - 1]);
            const float w0 = ex(m4, M);
            lt4 *= w0;
            orot4[0] *= w0;
            orot4[1] *= w0;
            for (int w = 1; w < np; ++w) {
                const float* xb = part(w);
                const float ww = ex(xb[XM + NHX - 1], M);
                lt4 = fmaf(ww, xb[XM + 2 * NHX - 1], lt4);
#pragma unroll
                for (int q = 0; q < 2; ++q) orot4[q] = fmaf(ww, xb[(NHX - 1) * kD + 16 * (4 * q + G) + n], orot4[q]);
            }
            if (l == 0) part(1)[XM + 3 * NHX - 1] = m4;
        }
        wave_sync();
#pragma unroll
        for (int hh = 0; hh < NHX; ++hh) {
            const float m0 = part(1)[XM + 2 * NHX + hh];
            float M = m0;
            for (int w = 1; w < np; ++w) M = fmaxf(M, part(w)[XM + hh]);
            const float w0 = ex(m0, M);
            oplain[hh][0] *= w0;
            oplain[hh][1] *= w0;
            for (int w = 1; w < np; ++w) {
                const float* xb = part(w);
                const float ww = ex(xb[XM + hh], M);
                const float2 y = *reinterpret_cast<const float2*>(xb + XP + hh * kD + 2 * l);
                oplain[hh][0] = fmaf(ww, y.x, oplain[hh][0]);
                oplain[hh][1] = fmaf(ww, y.y, oplain[hh][1]);
            }
        }
    }
    if (a.n_split == 1 || a.group > 1) {
        wave_sync();
#pragma unroll
        for (int hg = 0; hg < NH; ++hg) {
            if (4 * hg + G < g) {
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) sm.q[4 * hg + G][16 * mt + n] = orot[hg][mt];
                if (n == 0) sm.hv[4 * hg + G][3] = lt[hg];
            }
        }
        if constexpr (X1) {
#pragma unroll
            for (int q = 0; q < 2; ++q) sm.q[NHX - 1][16 * (4 * q + G) + n] = orot4[q];
            if (l == 0) sm.hv[NHX - 1][3] = lt4;
        }
        wave_sync();
        if (a.rotate) lds_hadamard<NHX>(sm.q, g);
        const float rs = a.rotate ? kInvSqrt128 : 1.f;
#pragma unroll
        for (int hh = 0; hh < NHX; ++hh) {
            if (hh < g) {
                const float L = sm.hv[hh][3];
                float o0 = sm.q[hh][2 * l] * rs + oplain[hh][0];
                float o1 = sm.q[hh][2 * l + 1] * rs + oplain[hh][1];
                o0 = L > 0.f ? o0 / L : 0.f;
                o1 = L > 0.f ? o1 / L : 0.f;
                const size_t idx = (qrow + hh) * kD + 2 * l;
                if (a.out_bf16)
                    reinterpret_cast<uint32_t*>(a.out)[idx >> 1] =
                        (uint32_t)f32_to_bf16(o0) | ((uint32_t)f32_to_bf16(o1) << 16);
                else
                    *reinterpret_cast<float2*>(static_cast<float*>(a.out) + idx) = make_float2(o0, o1);
            }
        }
    } else {
#pragma unroll
        for (int hg = 0; hg < NH; ++hg) {
            if (4 * hg + G < g) {
                float* P = a.ws + ((qrow + 4 * hg + G) * a.n_split + split) * kPart;
#pragma unroll
                for (int mt = 0; mt < 8; ++mt) P[4 + 16 * mt + n] = orot[hg][mt];
                if (n == 0) {
                    P[0] = m_run[hg];
                    P[1] = lt[hg];
                }
            }
        }
        if (X1 && g == NHX) {  // a chunk of a larger group may leave the extra head slot empty
            float* P = a.ws + ((qrow + NHX - 1) * a.n_split + split) * kPart;
#pragma unroll
            for (int q = 0; q < 2; ++q) P[4 + 16 * (4 * q + G) + n] = orot4[q];
            if (l == 0) {
                P[0] = m4;
                P[1] = lt4;
            }
        }
#pragma unroll
        for (int hh = 0; hh < NHX; ++hh) {
            if (hh < g) {
                float* P = a.ws + ((qrow + hh) * a.n_split + split) * kPart;
                *reinterpret_cast<float2*>(P + 132 + 2 * l) = make_float2(oplain[hh][0], oplain[hh][1]);
            }
        }
    }
}

// Merge of the split partials of a (sequence, query head): log-sum-exp weights, the inverse
// rotation of the body part in registers (lane l holds channels 2l, 2l + 1), normalisation.
// W waves per (sequence, query head), 256 threads per workgroup: W = 1 (four heads per
// workgroup) for few splits; W = 4 for many, wave w summing splits w, w + 4, ... and wave 0
// adding the four sums in a fixed order (eight waves per head measured slower at 37 splits).
constexpr int kMergeWide = 9;  // from this many splits on, four waves per head

// Channel partner c ^ (2 m) of lane l's two channels: the value of lane l ^ m.
template <int M>
__device__ __forceinline__ float lane_xor(float v, int l) {
    if constexpr (M == 1) return fdpp_x1(v);
    else if constexpr (M == 2) return fdpp_x2(v);
    else if constexpr (M == 16) {
        const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return __uint_as_float(((l >> 4) & 1) ? x[0] : x[1]);
    } else if constexpr (M == 32) {
        const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return __uint_as_float(l < 32 ? x[1] : x[0]);
    } else {
        return __shfl_xor(v, M);
    }
}
// One butterfly stage of stride 2 M between lanes l and l ^ M (both channels): the lower
// channel keeps a + b, the upper one a - b.
template <int M>
__device__ __forceinline__ void fwht_stage(float (&x)[2], int l) {
    const bool upper = (l & M) != 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const float p = lane_xor<M>(x[e], l);
        x[e] = upper ? p - x[e] : x[e] + p;
    }
}

template <int W>
__global__ __launch_bounds__(256) void k_decode_merge(DecodeArgs a) {
    static_assert(W == 1 || W == 4, "one or four waves per head");
    constexpr int HPB = 4 / W;          // heads per workgroup
    constexpr int U = W == 1 ? 8 : 16;  // splits with loads in flight per wave
    __shared__ float red[W > 1 ? W - 1 : 1][2 * kD + 2];
    const int l = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int part = wv % W;
    const size_t bh = (size_t)blockIdx.x * HPB + wv / W;
    // W > 1: one head per workgroup, so every wave leaves here or none does.
    if (bh >= (size_t)a.n_streams / a.n_kv * a.n_q) return;
    const float* P = a.ws + bh * a.n_split * kPart;
    const int S = a.n_split;
    // Log-sum-exp over this wave's splits, U of them with every load in flight (indices past the
    // last split are clamped, their values unused), the sums kept relative to the running
    // maximum M of the splits that hold a probability mass.
    float M = -INFINITY, L = 0.f, acc[2] = {0.f, 0.f}, pl[2] = {0.f, 0.f};
    for (int s0 = part; s0 < S; s0 += U * W) {
        float mm[U], ll[U];
        float2 ov[U], pv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float* Ps = P + (size_t)min(s0 + u * W, S - 1) * kPart;
            mm[u] = Ps[0];
            ll[u] = Ps[1];
            ov[u] = *reinterpret_cast<const float2*>(Ps + 4 + 2 * l);
            pv[u] = *reinterpret_cast<const float2*>(Ps + 132 + 2 * l);
        }
        float mb = M;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (s0 + u * W < S && ll[u] > 0.f) mb = fmaxf(mb, mm[u]);
        if (mb == -INFINITY) continue;  // no mass so far
        const float r = exp2f(M - mb);  // 0 while M is still -inf
        L *= r;
        acc[0] *= r;
        acc[1] *= r;
        pl[0] *= r;
        pl[1] *= r;
        M = mb;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (s0 + u * W < S && ll[u] > 0.f) {
                const float w = exp2f(mm[u] - M);
                L += w * ll[u];
                acc[0] += w * ov[u].x;
                acc[1] += w * ov[u].y;
                pl[0] += w * pv[u].x;
                pl[1] += w * pv[u].y;
            }
        }
    }
    if constexpr (W > 1) {
        // waves 1..W-1 hand (M, L, sums) to wave 0, which rescales them to the common maximum
        // and adds them in wave order
        if (part > 0) {
            float* rw = red[part - 1];
            *reinterpret_cast<float2*>(rw + 2 * l) = make_float2(acc[0], acc[1]);
            *reinterpret_cast<float2*>(rw + kD + 2 * l) = make_float2(pl[0], pl[1]);
            if (l == 0) {
                rw[2 * kD] = M;
                rw[2 * kD + 1] = L;
            }
        }
        __syncthreads();
        if (part > 0) return;
        float Mw[W - 1];
        float Mt = M;
#pragma unroll
        for (int w = 0; w < W - 1; ++w) {
            Mw[w] = red[w][2 * kD];
            Mt = fmaxf(Mt, Mw[w]);
        }
        if (Mt != -INFINITY) {
            const float r = exp2f(M - Mt);
            L *= r;
            acc[0] *= r;
            acc[1] *= r;
            pl[0] *= r;
            pl[1] *= r;
#pragma unroll
            for (int w = 0; w < W - 1; ++w) {
                const float rw = exp2f(Mw[w] - Mt);  // 0 for a wave without mass
                const float2 x = *reinterpret_cast<const float2*>(red[w] + 2 * l);
                const float2 y = *reinterpret_cast<const float2*>(red[w] + kD + 2 * l);
                acc[0] += rw * x.x;
                acc[1] += rw * x.y;
                pl[0] += rw * y.x;
                pl[1] += rw * y.y;
                L += rw * red[w][2 * kD + 1];
            }
        }
    }
    if (a.rotate) {  // H o_rot: butterflies of stride 1 (in the lane), 2, 4, ..., 64
        const float t = acc[0];
        acc[0] = t + acc[1];
        acc[1] = t - acc[1];
        fwht_stage<1>(acc, l);
        fwht_stage<2>(acc, l);
        fwht_stage<4>(acc, l);
        fwht_stage<8>(acc, l);
        fwht_stage<16>(acc, l);
        fwht_stage<32>(acc, l);
    }
    const float rs = a.rotate ? kInvSqrt128 : 1.f;
    float o[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        o[e] = acc[e] * rs + pl[e];
        o[e] = L > 0.f ? o[e] / L : 0.f;
    }
    const size_t idx = bh * kD + 2 * l;
    if (a.out_bf16)
        reinterpret_cast<uint32_t*>(a.out)[idx >> 1] = (uint32_t)f32_to_bf16(o[0]) | ((uint32_t)f32_to_bf16(o[1]) << 16);
    else
        *reinterpret_cast<float2*>(static_cast<float*>(a.out) + idx) = make_float2(o[0], o[1]);
}

template <int BITS, int GQ, int CMP>
hipError_t launch_cfg(const DecodeArgs& a, int batch, hipStream_t stream) {
    const int streams = batch * a.n_kv;
    // group mode: one workgroup of n_split waves per (stream, chunk); else one wave per workgroup
    const int wpg = a.group > 1 ? a.group : 1;
    const dim3 grid((unsigned)(streams * a.n_chunk * (a.group > 1 ? 1 : a.n_split))), block(64 * wpg);
    const bool pg = a.block_table != nullptr;
    if constexpr (GQ == 4) {
        const size_t lds = wpg * sizeof(Smem4<1, 0>);
        if (pg) hipLaunchKernelGGL((k_decode4<BITS, 1, CMP, 1, 0>), grid, block, lds, stream, a);
        else hipLaunchKernelGGL((k_decode4<BITS, 1, CMP, 0, 0>), grid, block, lds, stream, a);
    } else if constexpr (GQ == 5) {
        const size_t lds = wpg * sizeof(Smem4<1, 1>);
        if (pg) hipLaunchKernelGGL((k_decode4<BITS, 1, CMP, 1, 1>), grid, block, lds, stream, a);
        else hipLaunchKernelGGL((k_decode4<BITS, 1, CMP, 0, 1>), grid, block, lds, stream, a);
    } else if constexpr (GQ == 8) {
        const size_t lds = wpg * sizeof(Smem4<2, 0>);
        if (pg) hipLaunchKernelGGL((k_decode4<BITS, 2, CMP, 1, 0>), grid, block, lds, stream, a);
        else hipLaunchKernelGGL((k_decode4<BITS, 2, CMP, 0, 0>), grid, block, lds, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_split == 1 || a.group > 1) return e;
    const size_t heads = (size_t)batch * a.n_q;
    if (a.n_split >= kMergeWide)
        hipLaunchKernelGGL(k_decode_merge<4>, dim3((unsigned)heads), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL(k_decode_merge<1>, dim3((unsigned)((heads + 3) / 4)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

template <int BITS, int CMP>
hipError_t launch_bits(const DecodeArgs& a, int batch, hipStream_t stream) {
    if (a.g_chunk <= 4) return launch_cfg<BITS, 4, CMP>(a, batch, stream);
    if (a.g_chunk == 5) return launch_cfg<BITS, 5, CMP>(a, batch, stream);
    return launch_cfg<BITS, 8, CMP>(a, batch, stream);
}

}  // namespace

DecodePlan plan_decode(int batch, int n_kv, int n_q, int bits, int max_len, int n_sink, int max_blocks) {
    DecodePlan p;
    int nb = max_len > n_sink ? (max_len - n_sink) / kG : 0;
    if (nb > max_blocks) nb = max_blocks;
    p.max_blocks_used = nb;
    const int g = n_kv > 0 ? n_q / n_kv : 1;
    // Groups above 8 query heads go to the row-digit kernels in chunks of at most 8 heads (as
    // even as possible), one wave per chunk; the chunks of a stream read the same tiles.
    p.n_chunk = (g + 7) / 8;
    p.g_chunk = (g + p.n_chunk - 1) / p.n_chunk;
    const int gc = p.g_chunk;
    const int streams = batch * n_kv * p.n_chunk;  // waves per split
    // one wave per (split, chunk, stream).  Aim for one round of resident waves (the kernels'
    // occupancy on 1024 SIMDs), with at least 2 body tiles per split so that the per-wave
    // setup and the merge stay small against the streaming (measured on the Llama layer,
    // decode + merge: 1 tile per split 15.6 us, 2 tiles 14.1 us, 4 tiles 17.8 us).
    const int per_simd = gc <= 4 ? (bits == 2 ? 3 : 2) : 2;
    int want = (1024 * per_simd + streams - 1) / streams;
    // When kMaxGroup splits per stream already give every SIMD a wave, stop there: the splits
    // then merge inside their workgroup (no partials, no merge launch) and fewer, longer splits
    // spend less on per-split set-up, which beats filling the round (measured on 2-bit tiles,
    // 512 streams: 231 us instead of 242 at 32k tokens, 18-21 us instead of 23 at 1k; 256
    // streams: 123 us instead of 138 at 32k).
    const bool few = (long long)streams * kMaxGroup >= 1024;
    if (few && want > kMaxGroup) want = kMaxGroup;
    // Short streams there give one of those waves to the sink and residual chunks, which then run
    // beside the body tiles instead of after them, if the extra wave still fits the round (512
    // streams at 1k tokens: 17.9 us instead of 20.1, at 4k 39.4 instead of 41.3; from 8k on the
    // body splits gain more than that).
    const bool res_split = few && nb < kShortBody &&
                           (long long)streams * (std::min(want, kMaxGroup - 1) + 1) <= 1024LL * per_simd;
    if (res_split && want > kMaxGroup - 1) want = kMaxGroup - 1;
    if (want > nb / 2) want = nb / 2;
    p.n_res = 0;
    p.group = 0;
    if (want < 1 || (want == 1 && !res_split)) {
        p.n_split = 1;
        p.blocks_per_split = nb > 0 ? nb : 1;
        return p;
    }
    p.blocks_per_split = (nb + want - 1) / want;
    p.n_split = (nb + p.blocks_per_split - 1) / p.blocks_per_split;
    // A split stream is merged anyway: its sink + residual chunks (bf16, one memory round trip
    // each) get splits of their own, one per chunk a stream can hold, which run beside the body
    // splits -- when the extra waves still fit in the one round of resident waves (otherwise
    // body waves would wait for free slots behind them; measured: GQA-5 stress 28 % slower);
    // else one such split for all chunks if that fits.
    // (With kMaxGroup splits or fewer per stream the body splits share the chunks instead, unless
    // a short stream keeps a split for them, above.)
    const int chunks = (std::min(n_sink, std::max(max_len, 0)) + kRC - 1) / kRC + kG / kRC;
    if (few)
        p.n_res = res_split ? 1 : 0;
    else if ((long long)streams * (p.n_split + chunks) <= 1024LL * per_simd)
        p.n_res = chunks;
    else if ((long long)streams * (p.n_split + 1) <= 1024LL * per_simd)
        p.n_res = 1;
    p.n_split += p.n_res;
    // Up to kMaxGroup splits: the waves of one workgroup, merged there (no partials in memory,
    // no merge launch), when their LDS blocks fit the workgroup's 64 KB.
    const size_t blk = gc <= 4 ? sizeof(Smem4<1, 0>) : gc == 5 ? sizeof(Smem4<1, 1>) : sizeof(Smem4<2, 0>);
    if (p.n_split <= kMaxGroup && p.n_split * blk <= 65536) p.group = p.n_split;
    return p;
}

size_t decode_workspace_bytes(int batch, int n_q, const DecodePlan& plan) {
    if (plan.n_split == 1 || plan.group > 1) return 0;
    return (size_t)batch * n_q * plan.n_split * kPart * sizeof(float);
}

hipError_t launch_decode(const kvarn_cache& c, int bits, int compact, int rotate, int n_sink, int n_q, const void* q,
                         bool q_bf16, void* out, bool out_bf16, float sm_scale, const DecodePlan& plan, float* ws,
                         hipStream_t stream, const StepAppend* step) {
    DecodeArgs a;
    a.rotate = rotate;
    a.block_table = c.block_table;
    a.n_phys = c.n_phys;
    a.err_word = c.err_word;
    a.k_body = static_cast<const uint8_t*>(c.k_body);
    a.v_body = static_cast<const uint8_t*>(c.v_body);
    a.k_resid = static_cast<uint16_t*>(c.k_resid);
    a.v_resid = static_cast<uint16_t*>(c.v_resid);
    a.k_sink = static_cast<const uint16_t*>(c.k_sink);
    a.v_sink = static_cast<const uint16_t*>(c.v_sink);
    a.seq_len = c.seq_len;
    a.q = q;
    a.q_bf16 = q_bf16 ? 1 : 0;
    a.out = out;
    a.out_bf16 = out_bf16 ? 1 : 0;
    a.n_kv = c.n_kv;
    a.n_q = n_q;
    a.g = n_q / c.n_kv;
    a.max_blocks = c.max_blocks;
    a.n_sink = n_sink;
    a.scale_log2 = sm_scale * kLog2e;
    a.n_split = plan.n_split;
    a.bps = plan.blocks_per_split;
    a.n_res = plan.n_res;
    a.group = plan.group;
    a.n_streams = c.batch * c.n_kv;
    a.n_chunk = plan.n_chunk;
    a.g_chunk = plan.g_chunk;
    a.ws = ws;
    a.step_len = step ? step->len_before + 1 : 0;
    a.k_new = step ? static_cast<const uint16_t*>(step->k_new) : nullptr;
    a.v_new = step ? static_cast<const uint16_t*>(step->v_new) : nullptr;
    if (compact) return bits == 2 ? launch_bits<2, 1>(a, c.batch, stream) : launch_bits<4, 1>(a, c.batch, stream);
    return bits == 2 ? launch_bits<2, 0>(a, c.batch, stream) : launch_bits<4, 0>(a, c.batch, stream);
}

}  // namespace kvarn
