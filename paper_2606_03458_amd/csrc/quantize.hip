// KVarN tile quantizer for gfx950: Hadamard rotation (Sec. 2.2, App. A), VarN (App. H,
// Algorithm 1), asymmetric RTN (Sec. 2.1, Eq. 1) and bit-packing with the dual-scale aux of
// App. D.  One 256-thread workgroup quantizes one 128-token x 128-channel tile held entirely
// in registers: thread (tr, tc) owns tokens 8*tr..8*tr+7 and channels 8*tc..8*tc+7, with
// tc = lane % 16 (a DPP row of 16 lanes spans all 128 channels of a token) and
// tr = 4*wave + lane / 16.  Row (per-token) reductions stay inside a 16-lane row; column
// (per-channel) reductions cross the four 16-lane groups of a wave and then the four waves
// through LDS, in a fixed order so that every thread sees bit-identical results.
#include <type_traits>

#include "common.hpp"

namespace kvarn {
namespace {

constexpr int kThreads = 256;

struct QuantSmem {
    float red[2][4][kD];          // column partials [buffer][wave][channel]
    alignas(16) float tot[2][kD];  // column totals [buffer][channel]
    float rpick[4][4][8];         // row variances of each DPP row [wave][row][token], for the row update
    float rstat[2][4][2];         // per-wave row max / min [buffer][wave][max, min]
    alignas(16) uint8_t codes[kG * kD];  // keys: [token][channel]; values: [channel][token]
};

struct Lane {
    int tid, lane, wave, tc, tr;
    __device__ Lane() {
        tid = threadIdx.x;
        lane = tid & 63;
        wave = tid >> 6;
        tc = lane & 15;
        tr = wave * 4 + (lane >> 4);
    }
};

// ---- reductions ---------------------------------------------------------------------------
struct OpSum {
    __device__ static float f(float a, float b) { return a + b; }
};
// Max and min in the NaN-propagating forms: no operand here is a NaN (the input is finite), and
// fmaxf / fminf would first quiet every operand that comes from another lane or from LDS (one
// more instruction each).
__device__ __forceinline__ float fmax_any(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float fmin_any(float a, float b) { return __builtin_elementwise_minimum(a, b); }
struct OpMax {
    __device__ static float f(float a, float b) { return fmax_any(a, b); }
};
struct OpMin {
    __device__ static float f(float a, float b) { return fmin_any(a, b); }
};

template <int CTRL>
__device__ __forceinline__ float dppf(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Op over the 16 lanes of a DPP row: quad partners ^1 and ^2, then the other quad of the half
// (mirror within 8 lanes) and the other half (mirror within 16).  Each step combines two
// equal partial results, so every lane of the row ends with the same value.
template <class Op>
__device__ __forceinline__ float row16(float v) {
    v = Op::f(v, dppf<0xB1>(v));
    v = Op::f(v, dppf<0x4E>(v));
    v = Op::f(v, dppf<0x141>(v));
    return Op::f(v, dppf<0x140>(v));
}

// Op over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four rows of a wave).  With both operands equal,
// a row-pair swap returns (value of the even row, value of the odd row) in every lane of the
// pair, so all four lanes end with the same value.
template <class Op>
__device__ __forceinline__ float across_rows(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = Op::f(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return Op::f(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Across the 16 threads that share a channel block (all token blocks): the four rows of the
// wave, then the four waves through LDS.  Every thread of a channel block ends with the same
// values.
// With STAT, the same LDS round also carries one (max, min) pair per wave (xmax, xmin: the
// wave's values in, the workgroup's out).
// The four rows of the wave go as a reduce-scatter: permlane16_swap of two different values
// leaves, in every lane, the even-row and odd-row partials of one of them (rows 0, 2: the first,
// rows 1, 3: the second), and permlane32_swap of two such words the two half sums; the operands
// and their order are those of across_rows, so the sums are the same, but no lane computes
// results it then discards.  Row r of a wave ends with columns 8 tc + r and 8 tc + 4 + r.
template <class Op, bool STAT = false>
__device__ __forceinline__ void reduce_cols(float (&s)[8], QuantSmem& sm, int& buf, const Lane& L,
                                            float* xmax = nullptr, float* xmin = nullptr) {
    float t[4], rr[2];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(s[2 * p]), __float_as_uint(s[2 * p + 1]), false, false);
        t[p] = Op::f(__uint_as_float(x[0]), __uint_as_float(x[1]));
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const auto y = __builtin_amdgcn_permlane32_swap(__float_as_uint(t[2 * k]), __float_as_uint(t[2 * k + 1]), false, false);
        rr[k] = Op::f(__uint_as_float(y[0]), __uint_as_float(y[1]));
    }
    {
        const int r = L.lane >> 4;
        sm.red[buf][L.wave][8 * L.tc + r] = rr[0];
        sm.red[buf][L.wave][8 * L.tc + 4 + r] = rr[1];
    }
    if (STAT && L.lane == 0) {
        sm.rstat[buf][L.wave][0] = *xmax;
        sm.rstat[buf][L.wave][1] = *xmin;
    }
    __syncthreads();
    if (STAT) {
        *xmax = fmax_any(fmax_any(sm.rstat[buf][0][0], sm.rstat[buf][1][0]), fmax_any(sm.rstat[buf][2][0], sm.rstat[buf][3][0]));
        *xmin = fmin_any(fmin_any(sm.rstat[buf][0][1], sm.rstat[buf][1][1]), fmin_any(sm.rstat[buf][2][1], sm.rstat[buf][3][1]));
    }
    // each column's four wave partials are combined once (thread c of the first two waves),
    // then every thread of the channel block reads its eight totals
    if (L.tid < kD) {
        const int c = L.tid;
        sm.tot[buf][c] = Op::f(Op::f(Op::f(sm.red[buf][0][c], sm.red[buf][1][c]), sm.red[buf][2][c]), sm.red[buf][3][c]);
    }
    __syncthreads();
    const float4 lo = *reinterpret_cast<const float4*>(&sm.tot[buf][8 * L.tc]);
    const float4 hi = *reinterpret_cast<const float4*>(&sm.tot[buf][8 * L.tc + 4]);
    s[0] = lo.x; s[1] = lo.y; s[2] = lo.z; s[3] = lo.w;
    s[4] = hi.x; s[5] = hi.y; s[6] = hi.z; s[7] = hi.w;
    buf ^= 1;
}

// Across the 16 channel-block threads of a token row (one DPP row).
template <class Op>
__device__ __forceinline__ void reduce_rows(float (&s)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = row16<Op>(s[i]);
}

// Variance over tokens of every column of T*w (two-pass, ddof = 1).  The first LDS round also
// reduces the wave's (rmax, rmin) of the row variances to the workgroup's.
__device__ __forceinline__ void column_var(const float (&x)[8][8], const float (&w)[8], float (&var)[8],
                                           QuantSmem& sm, int& buf, const Lane& L, float& rmax, float& rmin) {
    // (explicit fmas: each pass forms x * w inside its own fma)
    float s[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = fmaf(x[i][j], w[i], acc);
        s[j] = acc;
    }
    reduce_cols<OpSum, true>(s, sm, buf, L, &rmax, &rmin);
    float mean[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) mean[j] = s[j] * (1.0f / kG);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float d = fmaf(x[i][j], w[i], -mean[j]);
            acc = fmaf(d, d, acc);
        }
        s[j] = acc;
    }
    reduce_cols<OpSum>(s, sm, buf, L);
#pragma unroll
    for (int j = 0; j < 8; ++j) var[j] = s[j] * (1.0f / (kG - 1));
}

// Variance over channels of every row of T*u (two-pass, ddof = 1).
__device__ __forceinline__ void row_var(const float (&x)[8][8], const float (&u)[8], float (&var)[8]) {
    float s[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = fmaf(x[i][j], u[j], acc);
        s[i] = acc;
    }
    reduce_rows<OpSum>(s);
    float mean[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) mean[i] = s[i] * (1.0f / kD);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float d = fmaf(x[i][j], u[j], -mean[i]);
            acc = fmaf(d, d, acc);
        }
        s[i] = acc;
    }
    reduce_rows<OpSum>(s);
#pragma unroll
    for (int i = 0; i < 8; ++i) var[i] = s[i] * (1.0f / (kD - 1));
}

// Imb of Algorithm 1 from the row variances (per token, replicated over tc) and the column
// variances (per channel, replicated over tr), in two parts: the wave's max / min of the row
// variances (reduced over the workgroup by column_var's first LDS round), then the value.
__device__ __forceinline__ void row_stat(const float (&vr)[8], float& rmax, float& rmin) {
    rmax = rmin = vr[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) {
        rmax = fmaxf(rmax, vr[k]);
        rmin = fminf(rmin, vr[k]);
    }
    rmax = across_rows<OpMax>(rmax);
    rmin = across_rows<OpMin>(rmin);
}
__device__ __forceinline__ float imbalance(float rmax, float rmin, const float (&vc)[8]) {
    float cmax = vc[0], cmin = vc[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) {
        cmax = fmaxf(cmax, vc[k]);
        cmin = fminf(cmin, vc[k]);
    }
    // all 128 channels live in one 16-lane row
    cmax = row16<OpMax>(cmax);
    cmin = row16<OpMin>(cmin);
    // (hardware reciprocal, ~1 ulp: Imb only ranks iterations, and values that close are ties)
    return rmax * __builtin_amdgcn_rcpf(fmaxf(rmin, 1e-8f)) + cmax * __builtin_amdgcn_rcpf(fmaxf(cmin, 1e-8f));
}

__device__ __forceinline__ float clampf(float v, float lo, float hi) { return fminf(fmaxf(v, lo), hi); }

// Natural log and exp on the hardware log2 / exp2.  Their arguments stay far from the denormal
// range (variances clamped to [var_min, var_max] >= 1e-30, log-scales to [log_lo, log_hi]
// within +-40), so no range fix-up is needed.
__device__ __forceinline__ float ln_hw(float v) { return __builtin_amdgcn_logf(v) * 0.6931471805599453f; }
__device__ __forceinline__ float exp_hw(float v) { return __builtin_amdgcn_exp2f(v * kLog2e); }

// ---- shared log-scale updates ----------------------------------------------------------------
// The four lanes of a wave that hold the same eight columns (lanes l, l^16, l^32, l^48) each
// update two of them, columns 2G and 2G + 1 of the eight (G = lane / 16); the sixteen lanes of
// a DPP row, which hold the same eight tokens, update token tc % 8.  The results are gathered
// back into every lane: with equal operands a 16-lane-row swap returns the (even row, odd row)
// values of a row pair and a half swap the (lower half, upper half) values; a DPP row
// broadcast returns lane i of the row.
__device__ __forceinline__ void gather_cols(const float (&own)[2], float (&out)[8]) {
    const auto a0 = __builtin_amdgcn_permlane16_swap(__float_as_uint(own[0]), __float_as_uint(own[0]), false, false);
    const auto a1 = __builtin_amdgcn_permlane16_swap(__float_as_uint(own[1]), __float_as_uint(own[1]), false, false);
    // a0 = (column 2*(G&2), column 2*(G&2) + 2), a1 = the same + 1; the half swap then gives the
    // values of rows 0-1 and 2-3
    const auto b0 = __builtin_amdgcn_permlane32_swap(a0[0], a0[0], false, false);  // columns 0, 4
    const auto b1 = __builtin_amdgcn_permlane32_swap(a0[1], a0[1], false, false);  // columns 2, 6
    const auto b2 = __builtin_amdgcn_permlane32_swap(a1[0], a1[0], false, false);  // columns 1, 5
    const auto b3 = __builtin_amdgcn_permlane32_swap(a1[1], a1[1], false, false);  // columns 3, 7
    out[0] = __uint_as_float(b0[0]); out[4] = __uint_as_float(b0[1]);
    out[2] = __uint_as_float(b1[0]); out[6] = __uint_as_float(b1[1]);
    out[1] = __uint_as_float(b2[0]); out[5] = __uint_as_float(b2[1]);
    out[3] = __uint_as_float(b3[0]); out[7] = __uint_as_float(b3[1]);
}
__device__ __forceinline__ void gather_rows(float own, float (&out)[8]) {
    out[0] = dppf<0x150>(own); out[1] = dppf<0x151>(own); out[2] = dppf<0x152>(own); out[3] = dppf<0x153>(own);
    out[4] = dppf<0x154>(own); out[5] = dppf<0x155>(own); out[6] = dppf<0x156>(own); out[7] = dppf<0x157>(own);
}
// v[2G + q] in lane row G (v the same in the four rows): a row-pair swap of two registers keeps
// the first one's even rows and moves the second one's even rows into the odd rows; a half swap
// of two registers keeps the first one's low half and moves the second one's low half up.
__device__ __forceinline__ float pick_col(const float (&v)[8], int q) {
    auto p16 = [](float a, float b) {
        return __uint_as_float(__builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false)[0]);
    };
    const float lo = p16(v[q], v[2 + q]), hi = p16(v[4 + q], v[6 + q]);  // rows: v[q], v[2+q], v[q], v[2+q]
    return __uint_as_float(__builtin_amdgcn_permlane32_swap(__float_as_uint(lo), __float_as_uint(hi), false, false)[0]);
}

// ---- narrow formats of the compact aux (App. D: 8-bit float scales, 16-bit float offset) ----
// OCP E4M3: 4-bit exponent with bias 7, 3-bit mantissa, subnormals m * 2^-9, largest 448.
// Grid value of x > 0 on the E4M3 grid of its binade (spacing 2^(e-3), 2^-9 below 2^-6),
// nearest with ties to even or upward, saturating at 448.  Scaling by powers of two is exact.
__device__ __forceinline__ float e4m3_round(float x, bool up) {
    if (x >= 448.f) return 448.f;
    int ex;
    frexpf(x, &ex);  // x in [2^(ex-1), 2^ex)
    const int E = max(ex - 1, -6);
    const float q = x * ldexpf(1.f, 3 - E);
    return (up ? ceilf(q) : rintf(q)) * ldexpf(1.f, E - 3);
}
// Byte of a value on the E4M3 grid (0 <= v <= 448).
__device__ __forceinline__ uint32_t e4m3_bits(float v) {
    if (v < 0.015625f) return (uint32_t)(v * 512.f);  // subnormal: m * 2^-9
    const uint32_t u = __float_as_uint(v);
    return ((((u >> 23) & 255u) - 120u) << 3) | ((u >> 20) & 7u);  // exponent - 127 + 7
}
// Nearest binary16 (ties to even), saturating at +-65504; returns the value and its bits.
__device__ __forceinline__ float fp16_round(float x, uint32_t& bits) {
    const _Float16 h = (_Float16)fminf(fmaxf(x, -65504.f), 65504.f);
    bits = __builtin_bit_cast(uint16_t, h);
    return (float)h;
}

// Quantize one tile.  src: token t at src + t*tstride elements, channels contiguous (16-byte
// aligned rows).  dst: the packed tile (16-byte aligned).
template <bool COMPACT, bool EXACT>
__device__ void quantize_tile(const void* src, bool bf16, int64_t tstride, int kind, const QParams& P, uint8_t* dst,
                              int32_t* best_out, QuantSmem& sm) {
    const Lane L;
    int buf = 0;
    float x[8][8];

    // ---- a1: load -------------------------------------------------------------------------
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t t = 8 * L.tr + i;
        if (bf16) {
            const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(src) + t * tstride + 8 * L.tc);
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                x[i][2 * k] = __uint_as_float(w[k] << 16);
                x[i][2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
            }
        } else {
            const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(src) + t * tstride + 8 * L.tc);
            const float4 a = p[0], b = p[1];
            x[i][0] = a.x; x[i][1] = a.y; x[i][2] = a.z; x[i][3] = a.w;
            x[i][4] = b.x; x[i][5] = b.y; x[i][6] = b.z; x[i][7] = b.w;
        }
    }

    // ---- a2: Hadamard along channels, butterflies of stride 1, 2, ..., 64 (not in the ablations
    // without rotation) ----------------------------------------------------------------------
    if (P.rotate) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int h = 1; h < 8; h <<= 1) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (!(j & h)) {
                        const float a = x[i][j], b = x[i][j + h];
                        x[i][j] = a + b;
                        x[i][j + h] = a - b;
                    }
                }
            }
        }
        // Cross-lane stages as one multiply-add each, x + p * B with B = +1 in the lower lane of
        // a pair and -1 in the upper one: the upper lane then holds -(a - b) instead of a - b.
        // Partners always hold values of the same sign, so the signs stay consistent and every
        // value is exactly +- the butterfly's (round to nearest is symmetric); after the four
        // stages lane tc holds (-1)^popcount(tc) times it, which the final scaling removes.
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) {  // channel stride 8*m lives in lane tc ^ m
            const float B = (L.tc & m) ? -1.f : 1.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    // partners ^1 and ^2 by DPP quad permutes, ^4 and ^8 through the LDS crossbar
                    const float p = m == 1 ? dppf<0xB1>(x[i][j]) : (m == 2 ? dppf<0x4E>(x[i][j]) : __shfl_xor(x[i][j], m));
                    x[i][j] = fmaf(p, B, x[i][j]);
                }
            }
        }
        const float scale = (__builtin_popcount(L.tc) & 1) ? -kInvSqrt128 : kInvSqrt128;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[i][j] *= scale;
        }
    }

    // ---- a3/a4: VarN (Algorithm 1), Cur = T * u[c] * w[t] with u = exp(-L_c), w = exp(-L_r) -
    // Each lane keeps the log-scales it updates (columns 2G, 2G + 1 and token tc % 8 of its
    // eight, current and best) and all eight scale factors u, w (gathered).
    const int G = L.lane >> 4, ir = L.tc & 7;
    float Lc2[2] = {0.f, 0.f}, bLc2[2] = {0.f, 0.f}, uo[2] = {1.f, 1.f};
    float Lr1 = 0.f, bLr1 = 0.f, wo = 1.f;
    float u[8], w[8], cv[8], rv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) u[k] = w[k] = 1.f;
    float rmax, rmin;
    row_var(x, u, rv);  // variance over channels of T's rows
    row_stat(rv, rmax, rmin);
    column_var(x, w, cv, sm, buf, L, rmax, rmin);  // variance over tokens of T's columns
    float I_best = imbalance(rmax, rmin, cv);
    int best = 0;
    for (int k = 1; k <= P.iters; ++k) {
        // column update from the current column variances u^2 * var_t(T w)
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const float v = clampf(uo[q] * uo[q] * pick_col(cv, q), P.var_min, P.var_max);
            Lc2[q] = clampf(Lc2[q] + 0.5f * ln_hw(v), P.log_lo, P.log_hi);
            uo[q] = exp_hw(-Lc2[q]);
        }
        gather_cols(uo, u);
        // row update from the row variances w^2 * var_c(T u)
        row_var(x, u, rv);
        {
            // the row's variances pass through LDS inside the wave to the lane that updates
            // token ir (LDS operations of a wave complete in order: no barrier)
            if (L.tc == 0) {
                *reinterpret_cast<float4*>(&sm.rpick[L.wave][G][0]) = make_float4(rv[0], rv[1], rv[2], rv[3]);
                *reinterpret_cast<float4*>(&sm.rpick[L.wave][G][4]) = make_float4(rv[4], rv[5], rv[6], rv[7]);
            }
            const float v = clampf(wo * wo * sm.rpick[L.wave][G][ir], P.var_min, P.var_max);
            Lr1 = clampf(Lr1 + 0.5f * ln_hw(v), P.log_lo, P.log_hi);
            wo = exp_hw(-Lr1);
        }
        gather_rows(wo, w);
        // imbalance of the new Cur; its column statistics seed the next column update
        float vr[8], vc[8];
#pragma unroll
        for (int m = 0; m < 8; ++m) vr[m] = w[m] * w[m] * rv[m];
        row_stat(vr, rmax, rmin);
        column_var(x, w, cv, sm, buf, L, rmax, rmin);
#pragma unroll
        for (int m = 0; m < 8; ++m) vc[m] = u[m] * u[m] * cv[m];
        const float I = imbalance(rmax, rmin, vc);
        if (I <= I_best) {  // later iteration wins ties
            I_best = I;
            best = k;
            bLc2[0] = Lc2[0];
            bLc2[1] = Lc2[1];
            bLr1 = Lr1;
        }
    }

    // ---- a5: balanced tile B = T / S_c* / S_r* ---------------------------------------------
    float Sc[8], Sr[8];
    {
        const float sc[2] = {exp_hw(bLc2[0]), exp_hw(bLc2[1])}, ui[2] = {exp_hw(-bLc2[0]), exp_hw(-bLc2[1])};
        gather_cols(sc, Sc);
        gather_cols(ui, u);
        gather_rows(exp_hw(bLr1), Sr);
        gather_rows(exp_hw(-bLr1), w);
    }
    float s2q[8];  // compact aux: the stored (E4M3) other-axis scale of this thread's rows/columns
    if constexpr (COMPACT) {
        // the other-axis scale is rounded first and the group RTN sees z = T / s2 (stored
        // value); the group-axis scale is absorbed exactly (RTN of a group ignores a common
        // factor)
#pragma unroll
        for (int m = 0; m < 8; ++m)
            s2q[m] = e4m3_round(clampf(kind == KVARN_KEYS ? Sr[m] : Sc[m], 0.015625f, 448.f), false);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[i][j] = x[i][j] / (kind == KVARN_KEYS ? s2q[i] : s2q[j]);
        }
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
#pragma unroll
            for (int j = 0; j < 8; ++j) x[i][j] = x[i][j] * u[j] * w[i];
        }
    }

    // ---- a6: RTN along the group axis (keys: per channel, values: per token) ----------------
    const float qmax = (float)((1 << P.bits) - 1);
    float mn[8], mx[8];
    if (kind == KVARN_KEYS) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            mn[j] = mx[j] = x[0][j];
#pragma unroll
            for (int i = 1; i < 8; ++i) {
                mn[j] = fminf(mn[j], x[i][j]);
                mx[j] = fmaxf(mx[j], x[i][j]);
            }
        }
        reduce_cols<OpMin>(mn, sm, buf, L);
        reduce_cols<OpMax>(mx, sm, buf, L);
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            mn[i] = mx[i] = x[i][0];
#pragma unroll
            for (int j = 1; j < 8; ++j) {
                mn[i] = fminf(mn[i], x[i][j]);
                mx[i] = fmaxf(mx[i], x[i][j]);
            }
        }
        reduce_rows<OpMin>(mn);
        reduce_rows<OpMax>(mx);
    }
    if constexpr (COMPACT) {
        // Both stored scales are E4M3 (at most 448) while their product is fixed by the data:
        // when the largest group step of the tile exceeds 448, a tile-wide 2^e moves from the
        // group scale into s2 (z / 2^e and s2 * 2^e leave every dequantized value unchanged,
        // and both products are exact), for the smallest such e >= 0 and no further than the
        // largest other-axis scale times 2^e stays within 448.  The shift needs every
        // other-axis scale at least 2^-6 (true unless log_lo is set below -4.1), so that s2 was
        // not clamped and scaling the stored s2 by 2^e equals storing 2^e times the scale.
        float st[3] = {0.f, 0.f, -__builtin_inff()};  // largest step, largest and -smallest other-axis scale
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const float so = kind == KVARN_KEYS ? Sr[m] : Sc[m];
            st[0] = fmaxf(st[0], (mx[m] - mn[m]) / qmax);
            st[1] = fmaxf(st[1], so);
            st[2] = fmaxf(st[2], -so);
        }
#pragma unroll
        for (int k = 0; k < 3; ++k) st[k] = across_rows<OpMax>(row16<OpMax>(st[k]));
        if (L.lane == 0) {
#pragma unroll
            for (int k = 0; k < 3; ++k) sm.red[buf][L.wave][k] = st[k];
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 3; ++k)
            st[k] = fmax_any(fmax_any(sm.red[buf][0][k], sm.red[buf][1][k]), fmax_any(sm.red[buf][2][k], sm.red[buf][3][k]));
        buf ^= 1;
        int e = 0;
        if (-st[2] >= 0.015625f)
            while (e < 64 && ldexpf(st[0], -e) > 448.f && ldexpf(st[1], e + 1) <= 448.f) ++e;
        if (e > 0) {
            const float down = ldexpf(1.f, -e), up = ldexpf(1.f, e);
#pragma unroll
            for (int m = 0; m < 8; ++m) {
                mn[m] *= down;
                mx[m] *= down;
                s2q[m] *= up;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
#pragma unroll
                for (int j = 0; j < 8; ++j) x[i][j] *= down;
            }
        }
    }
    // step and offset of each group: fp32 aux keeps them; the compact aux stores the step
    // rounded upward to E4M3 (the stored range covers the group) and the nearest binary16 of
    // the minimum, and the codes are chosen for those stored values
    float s[8], inv_s[8], off[8];
    uint32_t abits[8], bbits[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const float step = (mx[m] - mn[m]) / qmax;
        if constexpr (COMPACT) {
            s[m] = step == 0.f ? 1.f : e4m3_round(step, true);
            off[m] = fp16_round(mn[m], bbits[m]);
            abits[m] = e4m3_bits(s[m]);
        } else {
            s[m] = step == 0.f ? 1.f : step;
            off[m] = mn[m];
        }
        inv_s[m] = 1.0f / s[m];
    }
    // codes -> LDS (keys [t][c], values [c][t]), 8 bytes per thread per token / channel.
    // EXACT (unrotated and unbalanced tiles, the KIVI-style ablation, fp32 aux): the tile holds
    // the inputs themselves and a bf16 value can lie exactly halfway between two levels; the
    // quotient is then formed as qmax (x - mn) / (mx - mn) with one correctly rounded division,
    // which keeps such a value an exact half-integer, rounded half to even.  Otherwise the
    // reciprocal step is used.
    auto write_codes = [&](auto exact) {
        constexpr bool kExact = decltype(exact)::value;
        float den[8];
#pragma unroll
        for (int m = 0; m < 8; ++m) den[m] = mx[m] > mn[m] ? mx[m] - mn[m] : 1.f;
        // With fp32 aux the offset is the group minimum itself, so v - off >= 0 exactly, and at
        // the group maximum the quotient is qmax within a few ulps (correctly rounded step and
        // reciprocal, or division): rounding lands in [0, qmax] without a clamp.  The compact
        // aux rounds the offset to binary16 and the step up to E4M3, so its codes are clamped.
        // The code in the low byte of a word: u + 1.5 * 2^23 rounds u (0 <= u <= 15) to the
        // nearest integer, ties to even as rintf, into the low mantissa bits.
        auto code = [&](float v, int m) -> uint32_t {
            float u = kExact ? ((v - off[m]) * qmax) / den[m] : (v - off[m]) * inv_s[m];
            if constexpr (COMPACT) u = clampf(u, 0.f, qmax);  // (before rounding: the same codes)
            return __float_as_uint(u + 12582912.f);
        };
        // four such words -> their low bytes in order, by two byte permutes
        auto pack4 = [](uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
            return __builtin_amdgcn_perm(__builtin_amdgcn_perm(d, c, 0x0c0c0400u), __builtin_amdgcn_perm(b, a, 0x0c0c0400u),
                                         0x05040100u);
        };
        if (kind == KVARN_KEYS) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                uint32_t q[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) q[j] = code(x[i][j], j);
                *reinterpret_cast<uint2*>(&sm.codes[(8 * L.tr + i) * kD + 8 * L.tc]) =
                    make_uint2(pack4(q[0], q[1], q[2], q[3]), pack4(q[4], q[5], q[6], q[7]));
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                uint32_t q[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) q[i] = code(x[i][j], i);
                *reinterpret_cast<uint2*>(&sm.codes[(8 * L.tc + j) * kG + 8 * L.tr]) =
                    make_uint2(pack4(q[0], q[1], q[2], q[3]), pack4(q[4], q[5], q[6], q[7]));
            }
        }
    };
    write_codes(std::integral_constant<bool, EXACT>{});

    // ---- a7: aux (absorbed scales) --------------------------------------------------------
    float* aux = reinterpret_cast<float*>(dst + code_bytes(P.bits));
    uint8_t* caux = dst + code_bytes(P.bits);  // compact: b16[128] | a8[128] | s2_8[128]
    // group-axis values of 8 groups g0 .. g0 + 7 (a as E4M3 bytes, b as binary16), and the
    // other-axis s2 of 8 indices o0 .. o0 + 7
    auto put_group = [&](int g0) {
        *reinterpret_cast<uint4*>(caux + 2 * g0) =
            make_uint4(bbits[0] | bbits[1] << 16, bbits[2] | bbits[3] << 16, bbits[4] | bbits[5] << 16,
                       bbits[6] | bbits[7] << 16);
        *reinterpret_cast<uint2*>(caux + 256 + g0) =
            make_uint2(abits[0] | abits[1] << 8 | abits[2] << 16 | abits[3] << 24,
                       abits[4] | abits[5] << 8 | abits[6] << 16 | abits[7] << 24);
    };
    auto put_s2 = [&](int o0) {
        uint32_t sb[8];
#pragma unroll
        for (int m = 0; m < 8; ++m) sb[m] = e4m3_bits(s2q[m]);
        *reinterpret_cast<uint2*>(caux + 384 + o0) =
            make_uint2(sb[0] | sb[1] << 8 | sb[2] << 16 | sb[3] << 24, sb[4] | sb[5] << 8 | sb[6] << 16 | sb[7] << 24);
    };
    if constexpr (COMPACT) {
        if (kind == KVARN_KEYS) {
            if (L.tr == 0) put_group(8 * L.tc);  // per channel
            if (L.tc == 0) put_s2(8 * L.tr);     // per token
        } else {
            if (L.tc == 0) put_group(8 * L.tr);  // per token
            if (L.tr == 0) put_s2(8 * L.tc);     // per channel
        }
    } else {
      if (kind == KVARN_KEYS) {
        if (L.tr == 0) {  // per channel: a = s * S_c*, b = mn * S_c*
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                aux[8 * L.tc + j] = s[j] * Sc[j];
                aux[kD + 8 * L.tc + j] = mn[j] * Sc[j];
            }
        }
        if (L.tc == 0) {  // s2 per token
#pragma unroll
            for (int i = 0; i < 8; ++i) aux[2 * kD + 8 * L.tr + i] = Sr[i];
        }
    } else {
        if (L.tc == 0) {  // per token: a = s * S_r*, b = mn * S_r*
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                aux[8 * L.tr + i] = s[i] * Sr[i];
                aux[kD + 8 * L.tr + i] = mn[i] * Sr[i];
            }
        }
        if (L.tr == 0) {  // s2 per channel
#pragma unroll
            for (int j = 0; j < 8; ++j) aux[2 * kD + 8 * L.tc + j] = Sc[j];
        }
      }
    }
    if (best_out && L.tid == 0) *best_out = best;
    __syncthreads();

    // ---- a7: pack ------------------------------------------------------------------------------
    // Unit (sigma, lane L, w): its 16 codes e = 4s + q come from four 4-byte LDS reads d_s (byte
    // q = code e); code e goes to bit 8q + bits*(s % p) of word s / p, p = 8 / bits, so a word
    // is the OR of d_s shifted by bits*(s % p).  A 16-byte piece holds p units of one lane:
    // piece k of lane L in half sigma is stored at piece index 128*(bits/2)*sigma + 64*k + L, so
    // thread tid writes piece tid (and tid + 256 at 4 bits) and every store is contiguous.
    auto gather = [&](int sigma, int lanep, int wsel, uint32_t (&d)[4]) {
        const int m = lanep & 15, G4 = lanep >> 4;
        if (kind == KVARN_KEYS) {
            const int t = 64 * sigma + 16 * (wsel >> 1) + m;
            const int c0 = 64 * (wsel & 1) + 16 * G4;
            const uint4 v = *reinterpret_cast<const uint4*>(&sm.codes[t * kD + c0]);
            d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
        } else {
            const int c = 16 * wsel + m;
#pragma unroll
            for (int ss = 0; ss < 4; ++ss)
                d[ss] = *reinterpret_cast<const uint32_t*>(&sm.codes[c * kG + 64 * sigma + 16 * ss + 4 * G4]);
        }
    };
    if (P.bits == 2) {
        const int sigma = L.tid >> 7, k = (L.tid >> 6) & 1, lanep = L.tid & 63;
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t d[4];
            gather(sigma, lanep, 4 * k + i, d);
            w[i] = d[0] | (d[1] << 2) | (d[2] << 4) | (d[3] << 6);
        }
        reinterpret_cast<uint4*>(dst)[L.tid] = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
#pragma unroll
        for (int pi = 0; pi < 2; ++pi) {
            const int pc = L.tid + 256 * pi;
            const int sigma = pc >> 8, k = (pc >> 6) & 3, lanep = pc & 63;
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                uint32_t d[4];
                gather(sigma, lanep, 2 * k + i, d);
                w[2 * i] = d[0] | (d[1] << 4);
                w[2 * i + 1] = d[2] | (d[3] << 4);
            }
            reinterpret_cast<uint4*>(dst)[pc] = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
}

// Body tile blk of (sequence b, kv head kh) in the cache's tiles: dense [batch][n_kv][max_blocks],
// or paged (tile kh of pool block block_table[b][blk]).  -1 (and bit 1 of err_word) for a pool
// id outside [0, n_phys).
__device__ __forceinline__ int64_t body_tile(const kvarn_cache& c, int b, int kh, int blk) {
    if (!c.block_table) return ((int64_t)b * c.n_kv + kh) * c.max_blocks + blk;
    const int id = c.block_table[(size_t)b * c.max_blocks + blk];
    if (id < 0 || id >= c.n_phys) {
        if (threadIdx.x == 0 && c.err_word)
            __hip_atomic_fetch_or(c.err_word, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return -1;
    }
    return (int64_t)id * c.n_kv + kh;
}

struct TileArgs {
    QParams P;
    int kind;
    int x_bf16;
    const void* x;
    int64_t tile0, n_inner, x_outer, x_inner, x_token;
    uint8_t* out;
    int64_t out_outer, out_inner;
    int32_t* best_iter;
};

// Grids of many tiles: 4 waves per SIMD (128 VGPRs; the fp32-aux variants keep 8-12 values of
// the balance and RTN phase in scratch) hide the barrier and LDS latency of the reductions
// better than 3 (measured 11 % faster).  The flush, whose grids are one tile per stream and
// K/V, stays at 3 (4 measured slower there).
template <bool COMPACT, bool EXACT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_quantize_tiles(TileArgs a) {
    __shared__ QuantSmem sm;
    const int64_t tile = a.tile0 + blockIdx.x;
    const int64_t i = tile / a.n_inner, j = tile % a.n_inner;
    const size_t esz = a.x_bf16 ? 2 : 4;
    const char* src = static_cast<const char*>(a.x) + (size_t)(i * a.x_outer + j * a.x_inner) * esz;
    uint8_t* dst = a.out + (size_t)(i * a.out_outer + j * a.out_inner) * tile_bytes(a.P.bits, COMPACT);
    quantize_tile<COMPACT, EXACT>(src, a.x_bf16 != 0, a.x_token, a.kind, a.P, dst, a.best_iter ? a.best_iter + tile : nullptr,
                           sm);
}

struct FlushArgs {
    QParams P;
    kvarn_cache c;
    int n_sink;
};

// Runs after the append kernel has incremented seq_len: the tile (sequence, kv head, K|V) of a
// sequence whose residual just reached 128 tokens is quantized into body tile
// (len - n_sink)/128 - 1; nothing else is written.  Workgroup w owns tiles w, w + gridDim.x,
// ...: with one workgroup per tile (a flush known to be due for every sequence) that is one
// tile, and with a grid of resident size (due tiles unknown on the host) its 256 threads check
// up to 256 of its tiles at once and the workgroup quantizes the due ones, so that a call with
// few or no due tiles costs one round of short workgroups.
template <bool COMPACT, bool EXACT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3, 8))) void k_flush(FlushArgs a) {
    __shared__ QuantSmem sm;
    __shared__ uint64_t due_mask[kThreads / 64];
    // tile indices fit 32 bits: the host bounds batch * n_kv
    const int n = a.c.batch * a.c.n_kv * 2;
    const int step = (int)gridDim.x;
    // the body tile a due tile goes to, or -1 when it is not due (or the append refused it)
    auto target_block = [&](int t) -> int {
        const int b = (t >> 1) / a.c.n_kv;
        const int len = a.c.seq_len[b];
        if (len <= a.n_sink || (len - a.n_sink) % kG != 0) return -1;
        const int nb = (len - a.n_sink) / kG - 1;
        return nb < a.c.max_blocks ? nb : -1;
    };
    for (int base = (int)blockIdx.x; base < n; base += step * kThreads) {
        const int mine = base + (int)threadIdx.x * step;
        const bool due = mine < n && target_block(mine) >= 0;
        const uint64_t m = __ballot(due);
        __syncthreads();  // the previous round is done with due_mask and the tile state in sm
        if ((threadIdx.x & 63) == 0) due_mask[threadIdx.x >> 6] = m;
        __syncthreads();
        bool first = true;
        for (int w = 0; w < kThreads / 64; ++w) {
            // uniform across the workgroup: kept in scalar registers
            const uint64_t dm = due_mask[w];
            uint64_t mm = (uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)dm) |
                          (uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(dm >> 32)) << 32;
            for (; mm; mm &= mm - 1) {
                const int t = base + (64 * w + __builtin_ctzll(mm)) * step;
                const int kind = t & 1;
                const int stream = t >> 1;
                const int b = stream / a.c.n_kv;
                const int64_t ti = body_tile(a.c, b, stream % a.c.n_kv, target_block(t));
                if (ti < 0) continue;
                if (!first) __syncthreads();  // every thread is done with the previous tile's LDS
                first = false;
                const uint16_t* src =
                    static_cast<const uint16_t*>(kind ? a.c.v_resid : a.c.k_resid) + (size_t)stream * kG * kD;
                uint8_t* dst =
                    static_cast<uint8_t*>(kind ? a.c.v_body : a.c.k_body) + (size_t)ti * tile_bytes(a.P.bits, COMPACT);
                quantize_tile<COMPACT, EXACT>(src, true, kD, kind, a.P, dst, nullptr, sm);
            }
        }
    }
}

struct PrefillArgs {
    QParams P;
    kvarn_cache c;
    int n_sink;
    const void* k;
    const void* v;
    int x_bf16;
    const int32_t* cu;  // [batch + 1] prompt offsets (rows of k, v)
    int max_len;
    int groups;         // body tiles per (sequence, kv head) the grid covers
};

// Prompt length of sequence b, or -1 when it cannot be written (longer than the launch bound or
// than the body).
__device__ __forceinline__ int prefill_len(const PrefillArgs& a, int b) {
    const int L = a.cu[b + 1] - a.cu[b];
    const int nb = L > a.n_sink ? (L - a.n_sink) / kG : 0;
    return (L < 0 || L > a.max_len || nb > a.c.max_blocks) ? -1 : L;
}

// One workgroup per (sequence, kv head, K|V, body tile): quantizes the prompt's tile straight
// from the packed rows (token stride n_kv * 128 elements).
template <bool COMPACT, bool EXACT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_prefill_tiles(PrefillArgs a) {
    __shared__ QuantSmem sm;
    const int blk = (int)(blockIdx.x % a.groups);
    const int64_t rest = blockIdx.x / a.groups;
    const int kind = (int)(rest & 1);
    const int64_t stream = rest >> 1;
    const int b = (int)(stream / a.c.n_kv), kh = (int)(stream % a.c.n_kv);
    const int L = prefill_len(a, b);
    if (L < 0 || blk >= (L > a.n_sink ? (L - a.n_sink) / kG : 0)) return;
    const int64_t ti = body_tile(a.c, b, kh, blk);
    if (ti < 0) return;
    const size_t esz = a.x_bf16 ? 2 : 4;
    const int64_t row = (int64_t)a.cu[b] + a.n_sink + (int64_t)blk * kG;
    const char* src = static_cast<const char*>(kind ? a.v : a.k) + (size_t)((row * a.c.n_kv + kh) * kD) * esz;
    uint8_t* dst = static_cast<uint8_t*>(kind ? a.c.v_body : a.c.k_body) + (size_t)ti * tile_bytes(a.P.bits, COMPACT);
    quantize_tile<COMPACT, EXACT>(src, a.x_bf16 != 0, (int64_t)a.c.n_kv * kD, kind, a.P, dst, nullptr, sm);
}

// One workgroup per (sequence, kv head): sink and residual rows as bf16, then seq_len.
__global__ __launch_bounds__(kThreads) void k_prefill_copy(PrefillArgs a) {
    const int64_t stream = blockIdx.x;
    const int b = (int)(stream / a.c.n_kv), kh = (int)(stream % a.c.n_kv);
    const int L = prefill_len(a, b);
    if (threadIdx.x == 0 && kh == 0) {
        a.c.seq_len[b] = L < 0 ? 0 : L;
        if (L < 0 && a.c.err_word)
            __hip_atomic_fetch_or(a.c.err_word, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (L < 0) return;
    const int ns = min(L, a.n_sink);
    const int nr = L > a.n_sink ? (L - a.n_sink) % kG : 0;
    const int r0 = L - nr;  // first residual row of the prompt
    // rows [0, ns) -> sink, rows [r0, L) -> residual; 2 rows of 128 channels per pass
    for (int i = threadIdx.x; i < (ns + nr) * kD; i += kThreads) {
        const int t = i / kD, c = i % kD;
        const int row = t < ns ? t : r0 + (t - ns);
        const size_t at = ((size_t)(a.cu[b] + row) * a.c.n_kv + kh) * kD + c;
        uint16_t kb, vb;
        if (a.x_bf16) {
            kb = static_cast<const uint16_t*>(a.k)[at];
            vb = static_cast<const uint16_t*>(a.v)[at];
        } else {
            kb = f32_to_bf16(static_cast<const float*>(a.k)[at]);
            vb = f32_to_bf16(static_cast<const float*>(a.v)[at]);
        }
        if (t < ns) {
            const size_t o = ((size_t)stream * a.n_sink + t) * kD + c;
            static_cast<uint16_t*>(a.c.k_sink)[o] = kb;
            static_cast<uint16_t*>(a.c.v_sink)[o] = vb;
        } else {
            const size_t o = ((size_t)stream * kG + (t - ns)) * kD + c;
            static_cast<uint16_t*>(a.c.k_resid)[o] = kb;
            static_cast<uint16_t*>(a.c.v_resid)[o] = vb;
        }
    }
}

}  // namespace

// Unrotated, unbalanced tiles with fp32 aux (the KIVI-style ablation) take the quantizer variant
// whose RTN quotient keeps exact ties exact.
bool exact_quotient(const QParams& qp) { return !qp.compact && qp.iters == 0 && !qp.rotate; }

hipError_t launch_quantize_tiles(const QParams& qp, int kind, const void* x, bool x_bf16, int64_t n_outer,
                                 int64_t n_inner, int64_t x_outer, int64_t x_inner, int64_t x_token, void* out,
                                 int64_t out_outer, int64_t out_inner, int32_t* best_iter, hipStream_t stream) {
    const bool exact = exact_quotient(qp);
    const int64_t total = n_outer * n_inner;
    const int64_t kMaxGrid = 1 << 30;
    for (int64_t t0 = 0; t0 < total; t0 += kMaxGrid) {
        const int64_t n = total - t0 < kMaxGrid ? total - t0 : kMaxGrid;
        TileArgs a{qp, kind, x_bf16 ? 1 : 0, x, t0, n_inner, x_outer, x_inner, x_token,
                   static_cast<uint8_t*>(out), out_outer, out_inner, best_iter};
        if (qp.compact)
            hipLaunchKernelGGL((k_quantize_tiles<true, false>), dim3((unsigned)n), dim3(kThreads), 0, stream, a);
        else if (exact)
            hipLaunchKernelGGL((k_quantize_tiles<false, true>), dim3((unsigned)n), dim3(kThreads), 0, stream, a);
        else
            hipLaunchKernelGGL((k_quantize_tiles<false, false>), dim3((unsigned)n), dim3(kThreads), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_prefill(const QParams& qp, const kvarn_cache& c, int n_sink, const void* k, const void* v,
                          bool x_bf16, const int32_t* cu_seqlens, int max_len, hipStream_t stream) {
    const bool exact = exact_quotient(qp);
    int groups = max_len > n_sink ? (max_len - n_sink) / kG : 0;
    if (groups > c.max_blocks) groups = c.max_blocks;
    PrefillArgs a{qp, c, n_sink, k, v, x_bf16 ? 1 : 0, cu_seqlens, max_len, groups > 0 ? groups : 1};
    const int64_t streams = (int64_t)c.batch * c.n_kv;
    if (groups > 0) {
        const int64_t n = streams * 2 * groups;
        if (n >= (int64_t)1 << 31) return hipErrorInvalidValue;
        if (qp.compact)
            hipLaunchKernelGGL((k_prefill_tiles<true, false>), dim3((unsigned)n), dim3(kThreads), 0, stream, a);
        else if (exact)
            hipLaunchKernelGGL((k_prefill_tiles<false, true>), dim3((unsigned)n), dim3(kThreads), 0, stream, a);
        else
            hipLaunchKernelGGL((k_prefill_tiles<false, false>), dim3((unsigned)n), dim3(kThreads), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_prefill_copy, dim3((unsigned)streams), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_flush(const QParams& qp, const kvarn_cache& c, int n_sink, bool all_due, hipStream_t stream) {
    const bool exact = exact_quotient(qp);
    FlushArgs a{qp, c, n_sink};
    // resident grid: 256 CUs x 3 workgroups of 256 threads (the quantizer's occupancy)
    constexpr int64_t kResidentGrid = 768;
    const int64_t n = (int64_t)c.batch * c.n_kv * 2;
    const unsigned grid = (unsigned)(all_due ? n : (n < kResidentGrid ? n : kResidentGrid));
    if (qp.compact)
        hipLaunchKernelGGL((k_flush<true, false>), dim3(grid), dim3(kThreads), 0, stream, a);
    else if (exact)
        hipLaunchKernelGGL((k_flush<false, true>), dim3(grid), dim3(kThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((k_flush<false, false>), dim3(grid), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace kvarn
