/*
 * hccl_oracle.c -- plain CPU oracle for the collective semantics (TEST INFRASTRUCTURE).
 *
 * Only the test suite, the smoke entry point and the CPU-baseline leg of the benchmark use
 * this file. It shares nothing with the GPU library. It is deliberately slow and direct:
 * one element at a time, one contributor at a time, in the order the definitions state.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared
 * (-ffp-contract=off: an FP32 add is never fused with anything; on x86-64 float
 * arithmetic is SSE binary32 with round-to-nearest-even and no extended precision.)
 *
 * Citations are to the paper "HCCL: Collective Communication for Meta Training and
 * Inference Accelerators": Section II-A-2 (Near Memory Compute: copy and sum, BF16/FP16/FP32
 * operands, FP32 arithmetic, re-quantisation to the buffer type) and Section III-B-2 (Data
 * Path: the collectives AllReduce / ReduceScatter / AllGather / AllToAllv), Section IV-B-2
 * (device-resident collectives: AllToAllvDynamic, whose layout is read when it runs).
 */
#include "hccl_oracle.h"

#include <string.h>

/* ------------------------------------------------------------------------------------- */
/* Bit-level views                                                                        */
/* ------------------------------------------------------------------------------------- */

static uint32_t f32_bits(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return u;
}

static float bits_f32(uint32_t u) {
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* ------------------------------------------------------------------------------------- */
/* bfloat16: 1 sign bit, 8 exponent bits, 7 fraction bits -- the upper half of a binary32. */
/* ------------------------------------------------------------------------------------- */

/* Widening is exact: the 16 dropped bits are zero. */
float orc_bf16_to_f32(uint16_t h) { return bits_f32((uint32_t)h << 16); }

/*
 * Narrowing, round to nearest, ties to even. Keep the upper 16 bits (the truncated value
 * T) and look at the lower 16 bits (the remainder R, in units of 2^-16 of one bf16 ulp):
 * R above one half rounds up, R below rounds down, R exactly one half rounds to the T with
 * an even last bit. Rounding up carries into the exponent field when the fraction is all
 * ones, which is how the largest finite values round to infinity. A NaN stays a NaN: the
 * quiet bit is forced so that truncation cannot turn it into an infinity.
 */
uint16_t orc_f32_to_bf16(float f) {
    uint32_t u = f32_bits(f);
    uint32_t exp_field = (u >> 23) & 0xFFu;
    uint32_t frac = u & 0x7FFFFFu;
    uint32_t t = u >> 16;
    uint32_t r = u & 0xFFFFu;
    if (exp_field == 0xFFu && frac != 0) return (uint16_t)(t | 0x0040u);
    if (r > 0x8000u || (r == 0x8000u && (t & 1u))) t += 1u;
    return (uint16_t)t;
}

/* ------------------------------------------------------------------------------------- */
/* IEEE-754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.            */
/* ------------------------------------------------------------------------------------- */

float orc_f16_to_f32(uint16_t h) {
    uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
    uint32_t e = (h >> 10) & 0x1Fu;
    uint32_t m = h & 0x3FFu;
    if (e == 0x1Fu) {                       /* infinity or NaN */
        return bits_f32(sign | 0x7F800000u | (m << 13));
    }
    if (e == 0) {                           /* zero or subnormal: m * 2^-24, exact in fp32 */
        float v = (float)m * bits_f32(0x33800000u);   /* 2^-24 */
        return (sign ? -v : v);
    }
    /* normal: rebias the exponent from 15 to 127, widen the fraction from 10 to 23 bits */
    return bits_f32(sign | ((e - 15u + 127u) << 23) | (m << 13));
}

/*
 * Narrowing, round to nearest, ties to even, overflow to infinity, gradual underflow.
 * The binary32 value is (1.m) * 2^(e-127) for normal inputs. Its binary16 biased exponent
 * would be he = e - 127 + 15.
 *   he >= 31        : the value is at least 2^16 > the largest finite half -> infinity.
 *   1 <= he <= 30   : normal half; keep 10 of the 23 fraction bits and round on the other 13.
 *                     A round-up of an all-ones fraction carries into the exponent; from
 *                     he = 30 that gives the infinity encoding, as round-to-nearest requires.
 *   he <= 0         : subnormal half, counted in units of 2^-24. The 24-bit significand
 *                     (implicit one included) is shifted right by 14 - he bits and rounded on
 *                     the shifted-out bits. A carry out of the top gives the smallest normal.
 */
uint16_t orc_f32_to_f16(float f) {
    uint32_t u = f32_bits(f);
    uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
    int e = (int)((u >> 23) & 0xFFu);
    uint32_t m = u & 0x7FFFFFu;

    if (e == 0xFF) {                                    /* infinity or NaN */
        return (uint16_t)(sign | 0x7C00u | (m ? 0x0200u : 0u));
    }
    if (e == 0) return sign;                            /* fp32 zero/subnormal: < 2^-126, rounds to 0 */

    int he = e - 127 + 15;
    if (he >= 31) return (uint16_t)(sign | 0x7C00u);

    if (he >= 1) {
        uint32_t mant = m >> 13;
        uint32_t rem = m & 0x1FFFu;
        uint32_t r = ((uint32_t)he << 10) | mant;
        if (rem > 0x1000u || (rem == 0x1000u && (mant & 1u))) r += 1u;
        return (uint16_t)(sign | r);
    }

    uint32_t full = m | 0x800000u;                      /* 24-bit significand */
    int shift = 14 - he;                                /* >= 14 */
    if (shift > 24) return sign;                        /* below half of 2^-24 */
    uint32_t mant = full >> shift;
    uint32_t rem = full & ((1u << shift) - 1u);
    uint32_t half = 1u << (shift - 1);
    if (rem > half || (rem == half && (mant & 1u))) mant += 1u;
    return (uint16_t)(sign | mant);
}

void orc_f32_to_bf16_array(const float* in, uint16_t* out, size_t n) {
    for (size_t i = 0; i < n; ++i) out[i] = orc_f32_to_bf16(in[i]);
}

void orc_f32_to_f16_array(const float* in, uint16_t* out, size_t n) {
    for (size_t i = 0; i < n; ++i) out[i] = orc_f32_to_f16(in[i]);
}

void orc_f16_to_f32_array(const uint16_t* in, float* out, size_t n) {
    for (size_t i = 0; i < n; ++i) out[i] = orc_f16_to_f32(in[i]);
}

/* ------------------------------------------------------------------------------------- */
/* Element access                                                                         */
/* ------------------------------------------------------------------------------------- */

static int valid_dtype(int dtype) {
    return dtype == ORC_BF16 || dtype == ORC_FP16 || dtype == ORC_FP32 || dtype == ORC_INT32;
}

static size_t dtype_size(int dtype) {
    return (dtype == ORC_BF16 || dtype == ORC_FP16) ? 2u : 4u;
}

/* Read element i of a floating buffer and widen it to FP32 (exact for all three types). */
static float load_as_f32(const void* buf, int dtype, size_t i) {
    if (dtype == ORC_BF16) return orc_bf16_to_f32(((const uint16_t*)buf)[i]);
    if (dtype == ORC_FP16) return orc_f16_to_f32(((const uint16_t*)buf)[i]);
    return ((const float*)buf)[i];
}

/* Re-quantise an FP32 value to the buffer type and store it as element i. */
static void store_from_f32(void* buf, int dtype, size_t i, float v) {
    if (dtype == ORC_BF16) ((uint16_t*)buf)[i] = orc_f32_to_bf16(v);
    else if (dtype == ORC_FP16) ((uint16_t*)buf)[i] = orc_f32_to_f16(v);
    else ((float*)buf)[i] = v;
}

/* ------------------------------------------------------------------------------------- */
/* The reduction operator on one pair, FP32 and INT32.                                     */
/* ------------------------------------------------------------------------------------- */

/*
 * SUM is one binary32 addition (round to nearest even). MAX / MIN keep the running value
 * unless the new contributor is strictly larger / smaller; a NaN, once in the running
 * value, stays; a NaN contributor replaces a non-NaN running value.
 */
static float combine_f32(int op, float acc, float x) {
    if (op == ORC_SUM) return acc + x;
    if (acc != acc) return acc;
    if (x != x) return x;
    if (op == ORC_MAX) return (x > acc) ? x : acc;
    return (x < acc) ? x : acc;
}

/* SUM wraps modulo 2^32 (computed on unsigned values); MAX / MIN compare as signed. */
static int32_t combine_i32(int op, int32_t acc, int32_t x) {
    if (op == ORC_SUM) return (int32_t)((uint32_t)acc + (uint32_t)x);
    if (op == ORC_MAX) return (x > acc) ? x : acc;
    return (x < acc) ? x : acc;
}

/*
 * Reduce column i over the P contributors src[0..P-1] (each a buffer of the given type,
 * element index i) in the fixed order, and return the FP32 result before re-quantisation.
 *
 * group == 0: acc = x_0; acc = acc (+) x_1; ...; acc = acc (+) x_{P-1}.
 * group == L: for each group g of ranks gL .. gL+L-1, p_g is the same ascending fold over
 *             that group, kept in FP32; then acc = p_0 (+) p_1 (+) ... in ascending g.
 */
static float reduce_column_f32(int P, int dtype, int op, int group,
                               const void* const* src, size_t i) {
    if (group == 0) {
        float acc = load_as_f32(src[0], dtype, i);
        for (int r = 1; r < P; ++r) acc = combine_f32(op, acc, load_as_f32(src[r], dtype, i));
        return acc;
    }
    float total = 0.0f;
    for (int g = 0; g * group < P; ++g) {
        int first = g * group;
        float part = load_as_f32(src[first], dtype, i);
        for (int r = first + 1; r < first + group; ++r)
            part = combine_f32(op, part, load_as_f32(src[r], dtype, i));
        total = (g == 0) ? part : combine_f32(op, total, part);
    }
    return total;
}

static int32_t reduce_column_i32(int P, int op, int group, const void* const* src, size_t i) {
    if (group == 0) {
        int32_t acc = ((const int32_t*)src[0])[i];
        for (int r = 1; r < P; ++r) acc = combine_i32(op, acc, ((const int32_t*)src[r])[i]);
        return acc;
    }
    int32_t total = 0;
    for (int g = 0; g * group < P; ++g) {
        int first = g * group;
        int32_t part = ((const int32_t*)src[first])[i];
        for (int r = first + 1; r < first + group; ++r)
            part = combine_i32(op, part, ((const int32_t*)src[r])[i]);
        total = (g == 0) ? part : combine_i32(op, total, part);
    }
    return total;
}

static int check_reduce_args(int P, int dtype, int op, int group) {
    if (P < 1 || !valid_dtype(dtype)) return -1;
    if (op != ORC_SUM && op != ORC_MAX && op != ORC_MIN) return -1;
    if (group < 0) return -1;
    if (group > 0 && (P % group) != 0) return -1;
    return 0;
}

/* ------------------------------------------------------------------------------------- */
/* Other fold orders                                                                      */
/* ------------------------------------------------------------------------------------- */

/* Round an FP32 running value to the buffer type and widen it again. */
static float requantize(int dtype, float v) {
    if (dtype == ORC_BF16) return orc_bf16_to_f32(orc_f32_to_bf16(v));
    if (dtype == ORC_FP16) return orc_f16_to_f32(orc_f32_to_f16(v));
    return v;
}

static float comb_q(int op, int dtype, int requant, float acc, float x) {
    float v = combine_f32(op, acc, x);
    return requant ? requantize(dtype, v) : v;
}

/*
 * One element of shard `c` (or any shard for the orders that ignore it), folded in the
 * order `ord` describes. Returns the FP32 value before the final rounding.
 */
static float reduce_column_ordered_f32(int P, int dtype, int op, const orc_order* ord, int c,
                                       const void* const* src, size_t i) {
    int q = ord->requant;
    if (ord->kind == ORC_ORDER_RING) {
        int first = (c + 1) % P;
        float acc = load_as_f32(src[first], dtype, i);
        for (int k = 1; k < P; ++k) acc = comb_q(op, dtype, q, acc, load_as_f32(src[(first + k) % P], dtype, i));
        return acc;
    }
    if (ord->kind == ORC_ORDER_HALVING) {
        float v[512];
        for (int r = 0; r < P; ++r) v[r] = load_as_f32(src[r], dtype, i);
        for (int d = P / 2; d >= 1; d /= 2)
            for (int r = 0; r < d; ++r) v[r] = comb_q(op, dtype, q, v[r], v[r + d]);
        return v[0];
    }
    int group = (ord->kind == ORC_ORDER_TWO_LEVEL) ? ord->group : P;
    float total = 0.0f;
    for (int g = 0; g * group < P; ++g) {
        int first = g * group;
        float part = load_as_f32(src[first], dtype, i);
        for (int r = first + 1; r < first + group; ++r)
            part = comb_q(op, dtype, q, part, load_as_f32(src[r], dtype, i));
        total = (g == 0) ? part : comb_q(op, dtype, q, total, part);
    }
    return total;
}

static int32_t reduce_column_ordered_i32(int P, int op, const orc_order* ord, int c,
                                         const void* const* src, size_t i) {
    if (ord->kind == ORC_ORDER_RING) {
        int first = (c + 1) % P;
        int32_t acc = ((const int32_t*)src[first])[i];
        for (int k = 1; k < P; ++k) acc = combine_i32(op, acc, ((const int32_t*)src[(first + k) % P])[i]);
        return acc;
    }
    if (ord->kind == ORC_ORDER_HALVING) {
        int32_t v[512];
        for (int r = 0; r < P; ++r) v[r] = ((const int32_t*)src[r])[i];
        for (int d = P / 2; d >= 1; d /= 2)
            for (int r = 0; r < d; ++r) v[r] = combine_i32(op, v[r], v[r + d]);
        return v[0];
    }
    return reduce_column_i32(P, op, ord->kind == ORC_ORDER_TWO_LEVEL ? ord->group : 0, src, i);
}

static int check_order(int P, const orc_order* ord) {
    if (!ord) return -1;
    if (P > 512) return -1;
    if (ord->kind == ORC_ORDER_TWO_LEVEL && (ord->group < 1 || P % ord->group)) return -1;
    if (ord->kind == ORC_ORDER_HALVING && (P & (P - 1))) return -1;
    if (ord->kind < ORC_ORDER_ASCENDING || ord->kind > ORC_ORDER_HALVING) return -1;
    return 0;
}

/* ------------------------------------------------------------------------------------- */
/* Collectives                                                                            */
/* ------------------------------------------------------------------------------------- */

int orc_allreduce_ordered(int P, size_t count, int dtype, int op, const orc_order* ord,
                          const void* const* send, void* const* recv) {
    if (check_reduce_args(P, dtype, op, 0) != 0 || check_order(P, ord) != 0) return -1;
    if (ord->kind == ORC_ORDER_RING && ord->shard == 0) return -1;
    for (size_t i = 0; i < count; ++i) {
        int c = (ord->kind == ORC_ORDER_RING && ord->shard) ? (int)(i / ord->shard) : 0;
        if (dtype == ORC_INT32) {
            int32_t v = reduce_column_ordered_i32(P, op, ord, c, send, i);
            for (int r = 0; r < P; ++r) ((int32_t*)recv[r])[i] = v;
        } else {
            float v = reduce_column_ordered_f32(P, dtype, op, ord, c, send, i);
            for (int r = 0; r < P; ++r) store_from_f32(recv[r], dtype, i, v);
        }
    }
    return 0;
}

int orc_reduce_scatter_ordered(int P, size_t recvcount, int dtype, int op, const orc_order* ord,
                               const void* const* send, void* const* recv) {
    if (check_reduce_args(P, dtype, op, 0) != 0 || check_order(P, ord) != 0) return -1;
    size_t es = dtype_size(dtype);
    const void* block[512];
    for (int c = 0; c < P; ++c) {
        for (int r = 0; r < P; ++r) block[r] = (const char*)send[r] + (size_t)c * recvcount * es;
        for (size_t j = 0; j < recvcount; ++j) {
            if (dtype == ORC_INT32)
                ((int32_t*)recv[c])[j] = reduce_column_ordered_i32(P, op, ord, c, block, j);
            else
                store_from_f32(recv[c], dtype, j, reduce_column_ordered_f32(P, dtype, op, ord, c, block, j));
        }
    }
    return 0;
}

/*
 * AllReduce. Every output element is written only after all P inputs of that element have
 * been read, so an in-place call (recv[r] == send[r]) gives the same result.
 */
int orc_allreduce(int P, size_t count, int dtype, int op, int group,
                  const void* const* send, void* const* recv) {
    if (check_reduce_args(P, dtype, op, group) != 0) return -1;
    for (size_t i = 0; i < count; ++i) {
        if (dtype == ORC_INT32) {
            int32_t v = reduce_column_i32(P, op, group, send, i);
            for (int r = 0; r < P; ++r) ((int32_t*)recv[r])[i] = v;
        } else {
            float v = reduce_column_f32(P, dtype, op, group, send, i);
            for (int r = 0; r < P; ++r) store_from_f32(recv[r], dtype, i, v);
        }
    }
    return 0;
}

/* ReduceScatter: block c of every input, reduced, lands in recv[c]. */
int orc_reduce_scatter(int P, size_t recvcount, int dtype, int op, int group,
                       const void* const* send, void* const* recv) {
    if (check_reduce_args(P, dtype, op, group) != 0) return -1;
    size_t es = dtype_size(dtype);
    const void* block[512];
    if (P > 512) return -1;
    for (int c = 0; c < P; ++c) {
        for (int r = 0; r < P; ++r)
            block[r] = (const char*)send[r] + (size_t)c * recvcount * es;
        for (size_t j = 0; j < recvcount; ++j) {
            if (dtype == ORC_INT32)
                ((int32_t*)recv[c])[j] = reduce_column_i32(P, op, group, block, j);
            else
                store_from_f32(recv[c], dtype, j, reduce_column_f32(P, dtype, op, group, block, j));
        }
    }
    return 0;
}

/* AllGather: block q of every output is a byte copy of send[q]. */
int orc_allgather(int P, size_t sendcount, size_t elem_size,
                  const void* const* send, void* const* recv) {
    if (P < 1 || elem_size == 0) return -1;
    size_t bytes = sendcount * elem_size;
    for (int r = 0; r < P; ++r)
        for (int q = 0; q < P; ++q)
            if (bytes) memcpy((char*)recv[r] + (size_t)q * bytes, send[q], bytes);
    return 0;
}

/* AllToAllv: every (source, destination) block is a byte copy; nothing else is written. */
int orc_alltoallv(int P, size_t elem_size,
                  const void* const* send, const size_t* sendcounts, const size_t* sdispls,
                  void* const* recv, const size_t* recvcounts, const size_t* rdispls) {
    if (P < 1 || elem_size == 0) return -1;
    for (int s = 0; s < P; ++s)
        for (int d = 0; d < P; ++d)
            if (recvcounts[(size_t)d * P + s] != sendcounts[(size_t)s * P + d]) return -2;
    for (int s = 0; s < P; ++s) {
        for (int d = 0; d < P; ++d) {
            size_t n = sendcounts[(size_t)s * P + d];
            const char* from = (const char*)send[s] + sdispls[(size_t)s * P + d] * elem_size;
            char* to = (char*)recv[d] + rdispls[(size_t)d * P + s] * elem_size;
            for (size_t i = 0; i < n * elem_size; ++i) to[i] = from[i];
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------------------- */
/* AllToAllvDynamic (Section IV-B-2): layout from run-time metadata, then a plain AllToAllv */
/* ------------------------------------------------------------------------------------- */

/* A non-empty range [off, off + n) fits a buffer of `cap` rows. */
static int range_fits(int64_t off, int64_t n, size_t cap) {
    if (off < 0 || (uint64_t)off > cap) return 0;
    return (uint64_t)n <= cap - (uint64_t)off;
}

int orc_alltoallv_dynamic(int P, size_t elem_size, size_t row_elems,
                          const void* const* send, size_t send_cap, const int64_t* counts,
                          const int64_t* sdispls,
                          void* const* recv, size_t recv_cap, const int64_t* rdispls,
                          int64_t* recvcounts_out) {
    if (P < 1 || P > 64 || elem_size == 0 || row_elems == 0 || !counts) return -1;
    const size_t PP = (size_t)P * P;
    if (recvcounts_out)
        for (int s = 0; s < P; ++s)
            for (int d = 0; d < P; ++d) recvcounts_out[(size_t)d * P + s] = counts[(size_t)s * P + d];

    /* row offsets of every pair, send side [s*P+d], receive side [d*P+s] */
    int64_t sd[64 * 64], rd[64 * 64];
    for (size_t i = 0; i < PP; ++i)
        if (counts[i] < 0) return -2;
    for (int s = 0; s < P; ++s) {
        int64_t at = 0;  /* packed: destinations back to back, ascending */
        for (int d = 0; d < P; ++d) {
            const int64_t n = counts[(size_t)s * P + d];
            sd[(size_t)s * P + d] = sdispls ? sdispls[(size_t)s * P + d] : at;
            if (n > 0 && !range_fits(sd[(size_t)s * P + d], n, send_cap)) return -2;
            at += n;
        }
    }
    for (int d = 0; d < P; ++d) {
        int64_t at = 0;  /* packed: sources back to back, ascending */
        for (int s = 0; s < P; ++s) {
            const int64_t n = counts[(size_t)s * P + d];
            rd[(size_t)d * P + s] = rdispls ? rdispls[(size_t)d * P + s] : at;
            if (n > 0 && !range_fits(rd[(size_t)d * P + s], n, recv_cap)) return -2;
            at += n;
        }
        /* non-empty receive ranges of one destination are pairwise disjoint */
        for (int a = 0; a < P; ++a) {
            const int64_t na = counts[(size_t)a * P + d];
            if (na == 0) continue;
            for (int b = a + 1; b < P; ++b) {
                const int64_t nb = counts[(size_t)b * P + d];
                if (nb == 0) continue;
                const int64_t a0 = rd[(size_t)d * P + a], b0 = rd[(size_t)d * P + b];
                if (a0 < b0 + nb && b0 < a0 + na) return -2;
            }
        }
    }

    /* the layout is valid: move the data as an AllToAllv in elements */
    size_t sc[64 * 64], so[64 * 64], rc[64 * 64], ro[64 * 64];
    for (int s = 0; s < P; ++s)
        for (int d = 0; d < P; ++d) {
            const size_t n = (size_t)counts[(size_t)s * P + d] * row_elems;
            sc[(size_t)s * P + d] = n;
            rc[(size_t)d * P + s] = n;
            so[(size_t)s * P + d] = (size_t)sd[(size_t)s * P + d] * row_elems;
            ro[(size_t)d * P + s] = (size_t)rd[(size_t)d * P + s] * row_elems;
        }
    return orc_alltoallv(P, elem_size, send, sc, so, recv, rc, ro);
}
