/*
 * hccl_oracle.h -- plain CPU oracle for the collective semantics (TEST INFRASTRUCTURE).
 *
 * This header and hccl_oracle.c are the checker, not the product. Only the test suite,
 * the smoke entry point and the CPU-baseline leg of the benchmark may load or call them.
 * They share no code, header, table or helper with the GPU library: every conversion and
 * every fold below is written out again here on purpose.
 *
 * What is computed (paper: Section III-B-2 "Data Path" names the collectives, Section II-A-2
 * "Near Memory Compute" fixes the arithmetic):
 *   - element types BF16, FP16 and FP32 are reduced with FP32 arithmetic and re-quantised
 *     once to the buffer type (round to nearest, ties to even); INT32 is added with two's
 *     complement wrap-around.
 *   - the reduction visits contributors in a fixed order: ascending rank (group == 0), or
 *     the two-level order (group == L > 0): ranks are cut into consecutive groups of L,
 *     each group is folded in ascending rank order into an FP32 partial that is NOT
 *     re-quantised, then the partials are folded in ascending group order (rack-contiguous
 *     rank placement, Section V-D).
 *   - the accumulator is seeded with the first contributor itself (never with +0.0), so a
 *     column of negative zeros reduces to a negative zero.
 *
 * All buffers are host memory owned by the caller. Functions return 0 on success and a
 * negative value on a bad argument; they never abort.
 */
#ifndef HCCL_ORACLE_H
#define HCCL_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element types and reduction operators of the oracle (its own numbering). */
enum { ORC_BF16 = 0, ORC_FP16 = 1, ORC_FP32 = 2, ORC_INT32 = 3 };
enum { ORC_SUM = 0, ORC_MAX = 1, ORC_MIN = 2 };

/*
 * Fold orders beyond the default (paper: Section III-B-2 ring AllReduce; Section II-A-2: the
 * near-memory compute unit re-quantises every result to the buffer type).
 *   ORC_ORDER_ASCENDING : contributors 0, 1, ..., P-1.
 *   ORC_ORDER_TWO_LEVEL : `group` consecutive ranks folded ascending into a partial, then the
 *                         partials ascending.
 *   ORC_ORDER_RING      : the element belongs to shard c; contributors are visited
 *                         c+1, c+2, ..., P-1, 0, ..., c (the order a ring reduce-scatter adds
 *                         them as the partial travels towards its owner c). For all-reduce the
 *                         shard of element i is i / shard; for reduce-scatter it is the block.
 *   ORC_ORDER_HALVING   : recursive halving (P a power of two): level by level, value r is
 *                         combined with value r + d for d = P/2, P/4, ..., 1; the result is
 *                         value 0.
 * requant != 0: after every combine the running value is rounded to the buffer type and
 * widened again (no effect for FP32 and INT32).
 */
enum { ORC_ORDER_ASCENDING = 0, ORC_ORDER_TWO_LEVEL = 1, ORC_ORDER_RING = 2, ORC_ORDER_HALVING = 3 };

typedef struct {
    int kind;
    int group;       /* ORC_ORDER_TWO_LEVEL */
    size_t shard;    /* ORC_ORDER_RING, all-reduce: elements per shard */
    int requant;
} orc_order;

int orc_allreduce_ordered(int P, size_t count, int dtype, int op, const orc_order* order,
                          const void* const* send, void* const* recv);
int orc_reduce_scatter_ordered(int P, size_t recvcount, int dtype, int op, const orc_order* order,
                               const void* const* send, void* const* recv);

/* Scalar conversions, written from the IEEE-754 binary16 / bfloat16 definitions. */
float    orc_bf16_to_f32(uint16_t h);
uint16_t orc_f32_to_bf16(float f);
float    orc_f16_to_f32(uint16_t h);
uint16_t orc_f32_to_f16(float f);

/* Array forms of the conversions (used by the pins). */
void orc_f32_to_bf16_array(const float* in, uint16_t* out, size_t n);
void orc_f32_to_f16_array(const float* in, uint16_t* out, size_t n);
void orc_f16_to_f32_array(const uint16_t* in, float* out, size_t n);

/*
 * AllReduce: recv[r][i] = R(send[0][i], ..., send[P-1][i]) for every rank r and i < count.
 * recv[r] may equal send[r] (in place).
 */
int orc_allreduce(int P, size_t count, int dtype, int op, int group,
                  const void* const* send, void* const* recv);

/*
 * ReduceScatter: recv[c][j] = R(send[0][c*recvcount + j], ..., send[P-1][c*recvcount + j]).
 */
int orc_reduce_scatter(int P, size_t recvcount, int dtype, int op, int group,
                       const void* const* send, void* const* recv);

/* AllGather: recv[r][q*sendcount + j] = send[q][j] for every r, q and j < sendcount. */
int orc_allgather(int P, size_t sendcount, size_t elem_size,
                  const void* const* send, void* const* recv);

/*
 * AllToAllv: for every source s and destination d, the counts[s*P+d] elements that start at
 * element sdispls[s*P+d] of send[s] land at element rdispls[d*P+s] of recv[d]. Send arrays
 * are indexed [src*P + dst], receive arrays [dst*P + src]. recvcounts[d*P+s] must equal
 * sendcounts[s*P+d]. Receive elements outside every written range are left untouched.
 */
int orc_alltoallv(int P, size_t elem_size,
                  const void* const* send, const size_t* sendcounts, const size_t* sdispls,
                  void* const* recv, const size_t* recvcounts, const size_t* rdispls);

/*
 * AllToAllvDynamic (Section IV-B-2, device-resident collectives): an AllToAllv whose sizes, and
 * optionally offsets, are only known when it runs (a routing kernel writes them). Counts and
 * offsets are in rows of `row_elems` elements.
 *   counts[s*P + d]   rows source s sends to destination d
 *   sdispls[s*P + d]  row offset of that range in send[s]; NULL = packed: the ranges of one
 *                     source back to back in ascending destination order from row 0
 *   rdispls[d*P + s]  row offset in recv[d] of the rows from s; NULL = packed: ascending sources
 *   recvcounts_out[d*P + s] = counts[s*P + d], written whenever non-NULL (also on rejection)
 * Send buffers hold send_cap rows, receive buffers recv_cap rows. The layout is rejected
 * (return -2, no receive byte written) when a count is negative, a non-empty range does not lie
 * inside its buffer, or two non-empty receive ranges of one destination overlap. Ranges with
 * count 0 are not checked. Otherwise the rows move as orc_alltoallv moves elements.
 */
int orc_alltoallv_dynamic(int P, size_t elem_size, size_t row_elems,
                          const void* const* send, size_t send_cap, const int64_t* counts,
                          const int64_t* sdispls,
                          void* const* recv, size_t recv_cap, const int64_t* rdispls,
                          int64_t* recvcounts_out);

#ifdef __cplusplus
}
#endif
#endif
