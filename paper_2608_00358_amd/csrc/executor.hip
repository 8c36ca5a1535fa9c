// executor.hip -- the descriptor executor for gfx950 (MI355X).
//
// One launch runs one phase of a program (the single-GPU form of a work packet; paper, Section
// III-B-2). Every wavefront is an independent worker, the analogue of a message engine's
// control core (Section II-A-2: fetch the graph, evaluate dependencies, issue the work): it
// runs tile w of the phase when the grid has one wavefront per tile (a launch in which no tile
// waits), else tiles w, w + W, ... of a grid the CUs hold at once (or takes them by ticket on
// request), waits for each tile's dependencies, performs the copy or reduction of the tile
// with 128-bit coalesced loads and stores (the near-memory-compute analogue: FP32 arithmetic,
// one rounding to the buffer type), and signals completion with monotonically growing
// counters (the signal pairs of Section III-B-2). A launch may first wait on a trigger word (Section IV-B-3), and an AllToAllvDynamic
// step plans its layout on the device (Section IV-B-2).
//
// Memory model: dependency counters are written with agent-scope release and read with
// agent-scope acquire, so a consumer on another XCD (each XCD has its own L2) sees the
// producer's data. Programs without dependencies use no counters at all and nothing is shared
// between wavefronts.
#include <hip/hip_runtime.h>

#include <stddef.h>

#include <mutex>
#include <type_traits>

#include "program.h"

namespace hccl {

// Workspace of the allocation-free entry point: the program image, the dependency counters and
// the FP32 partials of one call live here instead of in memory the library allocates. Every
// device the library runs on holds its own copy, from the loading of this code object until
// the process ends. In host code `scratch` only names the symbol: its device address comes
// from workspace_address(), and only that address is ever handed to a kernel or a copy.
constexpr size_t kWorkspaceBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kWorkspaceBytes];

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWavesPerBlock = 4;
constexpr uint32_t kXcds = 8;  // XCDs of an MI355X
constexpr int kBlockThreads = kWavesPerBlock * kWaveSize;
#ifndef HCCL_SRC_BATCH
#define HCCL_SRC_BATCH 4
#endif
constexpr int kSrcBatch = HCCL_SRC_BATCH;  // sources whose loads are issued together

// 128-bit global accesses. Every byte of a collective is read once and written once, so the
// nontemporal hint streams it past the caches instead of evicting the program, the counters
// and other waves' lines. Copies store nontemporally too; reductions keep ordinary stores
// (measured faster for their small write share) unless they write many destinations (the
// two-level all-reduce's 64: half its traffic is stores, and streaming them measured 2 %
// faster).
#ifndef HCCL_NT_LOAD
#define HCCL_NT_LOAD 1
#endif
#ifndef HCCL_NT_STORE_COPY
#define HCCL_NT_STORE_COPY 1
#endif
#ifndef HCCL_NT_STORE_REDUCE
#define HCCL_NT_STORE_REDUCE 0
#endif
#ifndef HCCL_COPY_UNROLL
#define HCCL_COPY_UNROLL 4
#endif
#ifndef HCCL_REDUCE_UNROLL16
#define HCCL_REDUCE_UNROLL16 2
#endif

// Collective buffers are device memory (or pinned host memory), never LDS or scratch, so every
// data access goes through a global-address-space pointer. Through a generic pointer the same
// access compiles to a flat instruction, which also counts on the counter that scalar and LDS
// accesses use (a wait for a program-image read then waits for the data in flight as well)
// and needs a full 64-bit address per lane.
#define HCCL_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const HCCL_GLOBAL T* gp(const char* p) { return (const HCCL_GLOBAL T*)p; }
template <typename T>
__device__ __forceinline__ HCCL_GLOBAL T* gp(char* p) { return (HCCL_GLOBAL T*)p; }

__device__ __forceinline__ u32x4 vld(const char* p) {
    if constexpr (HCCL_NT_LOAD) return __builtin_nontemporal_load(gp<u32x4>(p));
    else return *gp<u32x4>(p);
}
// 16 bytes at an address aligned only to 4 or 2 bytes: one global_load_dwordx4 (global accesses
// of the HSA target may be unaligned). An ordinary load, not a non-temporal one: for these the
// non-temporal hint cost more than it saved (reduce-scatter of 8 ranks with a count that is not
// a multiple of 16 bytes: bf16 (2 Mi + 1) 63 -> 48 us, fp32 (1 Mi + 1) 68 -> 46 us while the
// inputs stay in the 256 MiB last-level cache; at 2 GiB of input bf16 462 -> 467 us, fp32
// 510 -> 467 us; AllToAllv of rows of 4 095 bf16 57 -> 46 us).
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x4_a2 __attribute__((ext_vector_type(4), aligned(2)));
template <int ES>
__device__ __forceinline__ u32x4 vld_shifted(const char* p) {
    typedef typename std::conditional<ES == 2, u32x4_a2, u32x4_a4>::type VU;
    return *gp<VU>(p);
}
// store of reduction results (NT: a step with many destinations)
template <bool NT = false>
__device__ __forceinline__ void vst(char* p, u32x4 v) {
    if constexpr (HCCL_NT_STORE_REDUCE || NT) __builtin_nontemporal_store(v, gp<u32x4>(p));
    else *gp<u32x4>(p) = v;
}
// destinations from which reduction results stream, and aligned copies write 8 KiB runs
constexpr uint32_t kWideStoreDsts = 8;
// store of copied data
__device__ __forceinline__ void vst_copy(char* p, u32x4 v) {
    if constexpr (HCCL_NT_STORE_COPY) __builtin_nontemporal_store(v, gp<u32x4>(p));
    else *gp<u32x4>(p) = v;
}

template <int DT> struct DtInfo;
template <> struct DtInfo<DT_BF16> { static constexpr int size = 2; typedef float acc; };
template <> struct DtInfo<DT_FP16> { static constexpr int size = 2; typedef float acc; };
template <> struct DtInfo<DT_FP32> { static constexpr int size = 4; typedef float acc; };
template <> struct DtInfo<DT_INT32> { static constexpr int size = 4; typedef int32_t acc; };

// ------------------------------------------------------------------ wave-uniform values
__device__ __forceinline__ uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ uint64_t uni64(uint64_t x) {
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// value held by lane j (j wave-uniform) of a lane-distributed 64-bit value
__device__ __forceinline__ uint64_t from_lane(uint64_t v, uint32_t j) {
    uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, j);
    uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), j);
    return ((uint64_t)hi << 32) | lo;
}

// uniform read of the program image through the constant address space (a scalar load)
template <typename T>
__device__ __forceinline__ T cld(const uint8_t* base, uint64_t off) {
    return *(const __attribute__((address_space(4))) T*)(base + off);
}
// the descriptor words run_tile decodes (little-endian, as on the host that packs them)
static_assert(offsetof(Desc, op) == 0 && offsetof(Desc, redop) == 1 && offsetof(Desc, flags) == 2 &&
                  offsetof(Desc, sig) == 3 && offsetof(Desc, nsrc) == 4 && offsetof(Desc, ndst) == 6 &&
                  offsetof(Desc, group) == 8 && offsetof(Desc, ndep) == 10 && offsetof(Desc, src) == 12 &&
                  offsetof(Desc, dst) == 16 && offsetof(Desc, dep) == 20 && offsetof(Desc, tile0) == 24 &&
                  offsetof(Desc, tile_elems) == 32 && offsetof(Desc, nelem) == 40 && offsetof(Desc, fold) == 48 &&
                  offsetof(Desc, requant) == 52 && offsetof(Desc, aux) == 56,
              "descriptor words");

__device__ __forceinline__ uint32_t elem_bytes(uint32_t dt) { return (dt == DT_BF16 || dt == DT_FP16) ? 2u : 4u; }

// ----------------------------------------------------------------------- conversions
// bf16 -> fp32 is exact: the bf16 bits are the upper half of the fp32 encoding.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest, ties to even: adding 0x7FFF plus the lowest kept bit to
// the encoding carries into the kept half exactly when the dropped half is above one half,
// or equal to one half with an odd kept half. NaNs keep sign and top payload, quiet bit set.
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float f16_lo(uint32_t w) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}
// fp32 -> fp16 with the hardware conversion in the default round-to-nearest-even mode
// (overflow to infinity, subnormal results kept).
__device__ __forceinline__ uint32_t f16_bits(float f) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
}

// --------------------------------------------------------------- reduction operators
// SUM: one binary32 addition (never fused). MAX / MIN: a NaN running value stays, a NaN
// contributor replaces a number, otherwise the strictly larger / smaller value wins.
template <int OPR>
__device__ __forceinline__ float comb(float a, float x) {
    if (OPR == RO_SUM) return a + x;
    if (a != a) return a;
    if (x != x) return x;
    if (OPR == RO_MAX) return (x > a) ? x : a;
    return (x < a) ? x : a;
}
template <int OPR>
__device__ __forceinline__ int32_t comb(int32_t a, int32_t x) {
    if (OPR == RO_SUM) return (int32_t)((uint32_t)a + (uint32_t)x);
    if (OPR == RO_MAX) return (x > a) ? x : a;
    return (x < a) ? x : a;
}

// ------------------------------------------------------- 8-element vectors per lane
template <int DT> struct Raw8 { u32x4 v[DtInfo<DT>::size / 2]; };

// SHIFT: p is aligned only to the element size
template <int DT, bool SHIFT = false>
__device__ __forceinline__ Raw8<DT> load8(const char* p) {
    Raw8<DT> r;
#pragma unroll
    for (int q = 0; q < DtInfo<DT>::size / 2; ++q)
        r.v[q] = SHIFT ? vld_shifted<DtInfo<DT>::size>(p + 16 * q) : vld(p + 16 * q);
    return r;
}

template <int DT, typename A>
__device__ __forceinline__ void widen8(const Raw8<DT>& r, A (&x)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if constexpr (DT == DT_BF16) {
            x[2 * i] = bf16_lo(r.v[0][i]);
            x[2 * i + 1] = bf16_hi(r.v[0][i]);
        } else if constexpr (DT == DT_FP16) {
            x[2 * i] = f16_lo(r.v[0][i]);
            x[2 * i + 1] = f16_hi(r.v[0][i]);
        } else if constexpr (DT == DT_FP32) {
            x[i] = __uint_as_float(r.v[0][i]);
            x[4 + i] = __uint_as_float(r.v[1][i]);
        } else {
            x[i] = (int32_t)r.v[0][i];
            x[4 + i] = (int32_t)r.v[1][i];
        }
    }
}

template <int DT, typename A, bool NT = false>
__device__ __forceinline__ void store8(char* p, const A (&x)[8]) {
    if constexpr (DT == DT_BF16 || DT == DT_FP16) {
        u32x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (DT == DT_BF16) w[i] = bf16_bits(x[2 * i]) | (bf16_bits(x[2 * i + 1]) << 16);
            else w[i] = f16_bits(x[2 * i]) | (f16_bits(x[2 * i + 1]) << 16);
        }
        vst<NT>(p, w);
    } else {
        u32x4 a, b;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (DT == DT_FP32) {
                a[i] = __float_as_uint(x[i]);
                b[i] = __float_as_uint(x[4 + i]);
            } else {
                a[i] = (uint32_t)x[i];
                b[i] = (uint32_t)x[4 + i];
            }
        }
        vst<NT>(p, a);
        vst<NT>(p + 16, b);
    }
}

// single elements (tails and misaligned operands)
template <int DT, typename A>
__device__ __forceinline__ A load1(const char* p) {
    if constexpr (DT == DT_BF16) return bf16_lo(*gp<uint16_t>(p));
    else if constexpr (DT == DT_FP16) return f16_lo(*gp<uint16_t>(p));
    else if constexpr (DT == DT_FP32) return *gp<float>(p);
    else return *gp<int32_t>(p);
}

template <int DT, typename A>
__device__ __forceinline__ void store1(char* p, A v) {
    if constexpr (DT == DT_BF16) *gp<uint16_t>(p) = (uint16_t)bf16_bits(v);
    else if constexpr (DT == DT_FP16) *gp<uint16_t>(p) = (uint16_t)f16_bits(v);
    else if constexpr (DT == DT_FP32) *gp<float>(p) = v;
    else *gp<int32_t>(p) = v;
}

// ---------------------------------------------------------------------------- REDUCE
struct TileOps {
    uint64_t src;     // lane j: address of source j at the tile's first element
    uint64_t dst;     // lane j: address of destination j at the tile's first element
    uint32_t nsrc, ndst, group;
    uint32_t fold = FOLD_LIST;
    uint32_t requant = 0;
};

// Re-quantisation of a partial to the destination type and back (Section II-A-2: the
// near-memory compute unit rounds every result to the buffer type).
template <int TO, bool REQ, typename A>
__device__ __forceinline__ A requant(A v) {
    if constexpr (REQ && TO == DT_BF16) return bf16_lo(bf16_bits(v));
    else if constexpr (REQ && TO == DT_FP16) return f16_lo(f16_bits(v));
    else return v;
}

template <int OPR, int TO, bool REQ, typename A>
__device__ __forceinline__ A combq(A a, A x) {
    return requant<TO, REQ>(comb<OPR>(a, x));
}

// Fold the sources of `count` elements starting at tile element `first`, one element per
// lane, contributors in list order (grouped when group > 0), and store to every destination.
template <int T0, int TR, int TO, int OPR, bool REQ = false>
__device__ __forceinline__ void reduce_elems(const TileOps& t, uint32_t first, uint32_t count, uint32_t lane) {
    typedef typename DtInfo<TO>::acc A;
    const uint32_t L = t.group ? t.group : t.nsrc;
    for (uint32_t e = first + lane; e < first + count; e += kWaveSize) {
        A tot = A(0);
        for (uint32_t g0 = 0; g0 < t.nsrc; g0 += L) {
            A part;
            const char* b0 = (const char*)from_lane(t.src, g0);
            if (g0 == 0) part = load1<T0, A>(b0 + (uint64_t)e * DtInfo<T0>::size);
            else part = load1<TR, A>(b0 + (uint64_t)e * DtInfo<TR>::size);
            const uint32_t gend = (g0 + L < t.nsrc) ? g0 + L : t.nsrc;
            for (uint32_t s = g0 + 1; s < gend; ++s) {
                const char* b = (const char*)from_lane(t.src, s);
                part = combq<OPR, TO, REQ>(part, load1<TR, A>(b + (uint64_t)e * DtInfo<TR>::size));
            }
            tot = (g0 == 0) ? part : combq<OPR, TO, REQ>(tot, part);
        }
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* b = (char*)from_lane(t.dst, j);
            store1<TO, A>(b + (uint64_t)e * DtInfo<TO>::size, tot);
        }
    }
}

// U vectors of 8 elements per lane: elements [base, base + U*512) of the tile, all in range.
// The destinations are 16-byte aligned at element base; SHIFT: the sources need not be.
template <int T0, int TR, int TO, int OPR, int U, bool REQ = false, bool SHIFT = false>
__device__ __forceinline__ void reduce_block(const TileOps& t, uint32_t base, uint32_t lane) {
    typedef typename DtInfo<TO>::acc A;
    // a first source of another type (a chained step's FP32 partial) needs its own registers
    constexpr bool kMixed = (T0 != TR);
    constexpr int SB = kMixed ? kSrcBatch / 2 : kSrcBatch;
    const uint32_t L = t.group ? t.group : t.nsrc;
    A tot[U][8], part[U][8];
    for (uint32_t g0 = 0; g0 < t.nsrc; g0 += L) {
        const uint32_t gend = (g0 + L < t.nsrc) ? g0 + L : t.nsrc;
        // Sources are visited in batches; every load of a batch is issued before the first
        // of them is folded, so one memory round trip serves the whole batch.
        for (uint32_t s = g0; s < gend; s += SB) {
            Raw8<T0> raw0[kMixed ? U : 1];
            Raw8<TR> raw[SB][U];
            const bool first_mixed = kMixed && s == 0;  // source 0 is typed T0
            if constexpr (kMixed) {
                if (first_mixed) {
                    const char* b = (const char*)from_lane(t.src, 0);
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        uint32_t e = base + ((uint32_t)u * kWaveSize + lane) * kVecElems;
                        raw0[u] = load8<T0, SHIFT>(b + (uint64_t)e * DtInfo<T0>::size);
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                if ((j > 0 || !first_mixed) && s + j < gend) {
                    const char* b = (const char*)from_lane(t.src, s + j);
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        uint32_t e = base + ((uint32_t)u * kWaveSize + lane) * kVecElems;
                        raw[j][u] = load8<TR, SHIFT>(b + (uint64_t)e * DtInfo<TR>::size);
                    }
                }
            }
            if constexpr (kMixed) {
                if (first_mixed) {
#pragma unroll
                    for (int u = 0; u < U; ++u) widen8<T0, A>(raw0[u], part[u]);
                }
            }
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                if ((j > 0 || !first_mixed) && s + j < gend) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        A x[8];
                        widen8<TR, A>(raw[j][u], x);
                        if (s + j == g0) {
#pragma unroll
                            for (int i = 0; i < 8; ++i) part[u][i] = x[i];
                        } else {
#pragma unroll
                            for (int i = 0; i < 8; ++i) part[u][i] = combq<OPR, TO, REQ>(part[u][i], x[i]);
                        }
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                tot[u][i] = (g0 == 0) ? part[u][i] : combq<OPR, TO, REQ>(tot[u][i], part[u][i]);
    }
    if (t.ndst >= kWideStoreDsts) {
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* b = (char*)from_lane(t.dst, j);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                uint32_t e = base + ((uint32_t)u * kWaveSize + lane) * kVecElems;
                store8<TO, A, true>(b + (uint64_t)e * DtInfo<TO>::size, tot[u]);
            }
        }
    } else {
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* b = (char*)from_lane(t.dst, j);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                uint32_t e = base + ((uint32_t)u * kWaveSize + lane) * kVecElems;
                store8<TO, A>(b + (uint64_t)e * DtInfo<TO>::size, tot[u]);
            }
        }
    }
}

// Elements [base, n) of the tile in vector steps (destinations 16-byte aligned at base), then
// single elements.
template <int T0, int TR, int TO, int OPR, bool REQ, bool SHIFT>
__device__ __forceinline__ void reduce_vectors(const TileOps& t, uint32_t base, uint32_t n, uint32_t lane) {
    constexpr int U = (DtInfo<TR>::size == 2) ? HCCL_REDUCE_UNROLL16 : 1;
    constexpr uint32_t kBlock = (uint32_t)U * kWaveSize * kVecElems;
    for (; base + kBlock <= n; base += kBlock) reduce_block<T0, TR, TO, OPR, U, REQ, SHIFT>(t, base, lane);
    // remaining whole 512-element steps, then single elements
    for (; base + kWaveSize * kVecElems <= n; base += kWaveSize * kVecElems)
        reduce_block<T0, TR, TO, OPR, 1, REQ, SHIFT>(t, base, lane);
    if (base < n) {
        // lanes whose 8 elements are all in range take one more vector step
        const uint32_t whole = (n - base) / kVecElems;
        if (lane < whole) reduce_block<T0, TR, TO, OPR, 1, REQ, SHIFT>(t, base, lane);
        base += whole * kVecElems;
    }
    if (base < n) reduce_elems<T0, TR, TO, OPR, REQ>(t, base, n - base, lane);
}

// A tile whose operands are not all 16-byte aligned keeps the vector steps when its
// destinations agree modulo 16 (a reduce-scatter of a count that is not a multiple of 16 bytes:
// every source of a block at one offset, the output at another): after a head of single
// elements the destinations are aligned, and the sources are read with 16-byte loads at their
// element alignment, folded in the same order. Otherwise element by element.
template <int T0, int TR, int TO, int OPR, bool REQ = false>
__device__ __forceinline__ void reduce_tile(const TileOps& t, uint32_t n, bool aligned, uint32_t lane) {
    if (aligned) {
        reduce_vectors<T0, TR, TO, OPR, REQ, false>(t, 0, n, lane);
        return;
    }
    const uint32_t dmis = (uint32_t)(from_lane(t.dst, 0) & 15u);
    if (__ballot(lane < t.ndst && (uint32_t)(t.dst & 15u) != dmis) != 0ull) {
        reduce_elems<T0, TR, TO, OPR, REQ>(t, 0, n, lane);
        return;
    }
    uint32_t head = ((16u - dmis) & 15u) / DtInfo<TO>::size;
    if (head > n) head = n;
    if (head) reduce_elems<T0, TR, TO, OPR, REQ>(t, 0, head, lane);
    reduce_vectors<T0, TR, TO, OPR, REQ, true>(t, head, n, lane);
}

// ------------------------------------------------------------- binary-tree (pairwise) fold
// The sources form the leaves of a complete binary tree in list order: (s0 s1) (s2 s3) ...,
// then pairs of those, up to the root (the recursive-halving order once the compiler has
// listed the ranks by bit reversal). Leaf k joins the pending subtree on each level where
// bit `level` of k is set; the pending subtrees live in a six-level stack (64 sources).
constexpr int kTreeLevels = 6;    // 2^6 = 64 sources
constexpr int kTreeBatch = 4;     // sources whose loads are issued together in a tree fold

template <int T, int OPR, bool REQ>
__device__ __forceinline__ void reduce_elems_tree(const TileOps& t, uint32_t first, uint32_t count, uint32_t lane) {
    typedef typename DtInfo<T>::acc A;
    for (uint32_t e = first + lane; e < first + count; e += kWaveSize) {
        A stk[kTreeLevels], root = A(0);
        for (uint32_t k = 0; k < t.nsrc; ++k) {
            const char* b = (const char*)from_lane(t.src, k);
            A v = load1<T, A>(b + (uint64_t)e * DtInfo<T>::size);
            bool placed = false;
#pragma unroll
            for (int l = 0; l < kTreeLevels; ++l) {
                if (!placed) {
                    if ((k >> l) & 1u) {
                        v = combq<OPR, T, REQ>(stk[l], v);
                    } else {
                        stk[l] = v;
                        placed = true;
                    }
                }
            }
            if (!placed) root = v;  // leaf 63 closes the 64-source tree
        }
#pragma unroll
        for (int l = 0; l < kTreeLevels; ++l)
            if ((1u << l) == t.nsrc) root = stk[l];
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* b = (char*)from_lane(t.dst, j);
            store1<T, A>(b + (uint64_t)e * DtInfo<T>::size, root);
        }
    }
}

template <int T, int OPR, bool REQ, bool SHIFT = false>
__device__ __forceinline__ void reduce_block_tree(const TileOps& t, uint32_t base, uint32_t lane) {
    typedef typename DtInfo<T>::acc A;
    A stk[kTreeLevels][8], root[8];
    const uint32_t e = base + lane * kVecElems;
    for (uint32_t s = 0; s < t.nsrc; s += kTreeBatch) {
        Raw8<T> raw[kTreeBatch];
#pragma unroll
        for (int j = 0; j < kTreeBatch; ++j) {
            if (s + j < t.nsrc) {
                const char* b = (const char*)from_lane(t.src, s + j);
                raw[j] = load8<T, SHIFT>(b + (uint64_t)e * DtInfo<T>::size);
            }
        }
#pragma unroll
        for (int j = 0; j < kTreeBatch; ++j) {
            if (s + j < t.nsrc) {
                const uint32_t k = s + j;
                A v[8];
                widen8<T, A>(raw[j], v);
                bool placed = false;
#pragma unroll
                for (int l = 0; l < kTreeLevels; ++l) {
                    if (!placed) {
                        if ((k >> l) & 1u) {
#pragma unroll
                            for (int i = 0; i < 8; ++i) v[i] = combq<OPR, T, REQ>(stk[l][i], v[i]);
                        } else {
#pragma unroll
                            for (int i = 0; i < 8; ++i) stk[l][i] = v[i];
                            placed = true;
                        }
                    }
                }
                if (!placed) {
#pragma unroll
                    for (int i = 0; i < 8; ++i) root[i] = v[i];
                }
            }
        }
    }
#pragma unroll
    for (int l = 0; l < kTreeLevels; ++l)
        if ((1u << l) == t.nsrc)
#pragma unroll
            for (int i = 0; i < 8; ++i) root[i] = stk[l][i];
    for (uint32_t j = 0; j < t.ndst; ++j) {
        char* b = (char*)from_lane(t.dst, j);
        store8<T, A>(b + (uint64_t)e * DtInfo<T>::size, root);
    }
}

template <int T, int OPR, bool REQ, bool SHIFT>
__device__ __forceinline__ void tree_vectors(const TileOps& t, uint32_t base, uint32_t n, uint32_t lane) {
    for (; base + kWaveSize * kVecElems <= n; base += kWaveSize * kVecElems)
        reduce_block_tree<T, OPR, REQ, SHIFT>(t, base, lane);
    if (base < n) {
        const uint32_t whole = (n - base) / kVecElems;
        if (lane < whole) reduce_block_tree<T, OPR, REQ, SHIFT>(t, base, lane);
        base += whole * kVecElems;
    }
    if (base < n) reduce_elems_tree<T, OPR, REQ>(t, base, n - base, lane);
}

// Operands not all 16-byte aligned: as reduce_tile, shifted source loads after a head of single
// elements when the destinations agree modulo 16, else element by element.
template <int T, int OPR, bool REQ>
__device__ __forceinline__ void reduce_tile_tree(const TileOps& t, uint32_t n, bool aligned, uint32_t lane) {
    if (aligned) {
        tree_vectors<T, OPR, REQ, false>(t, 0, n, lane);
        return;
    }
    const uint32_t dmis = (uint32_t)(from_lane(t.dst, 0) & 15u);
    if (__ballot(lane < t.ndst && (uint32_t)(t.dst & 15u) != dmis) != 0ull) {
        reduce_elems_tree<T, OPR, REQ>(t, 0, n, lane);
        return;
    }
    uint32_t head = ((16u - dmis) & 15u) / DtInfo<T>::size;
    if (head > n) head = n;
    if (head) reduce_elems_tree<T, OPR, REQ>(t, 0, head, lane);
    tree_vectors<T, OPR, REQ, true>(t, head, n, lane);
}

template <int T0, int TR, int TO>
__device__ __forceinline__ void reduce_dispatch_op(uint32_t op, const TileOps& t, uint32_t n, bool aligned, uint32_t lane) {
    if (op == RO_SUM) reduce_tile<T0, TR, TO, RO_SUM>(t, n, aligned, lane);
    else if constexpr (T0 == TR && TR == TO) {
        if (op == RO_MAX) reduce_tile<T0, TR, TO, RO_MAX>(t, n, aligned, lane);
        else reduce_tile<T0, TR, TO, RO_MIN>(t, n, aligned, lane);
    }
}

template <int T>
__device__ __forceinline__ void run_tree(uint32_t op, const TileOps& t, uint32_t n, bool aligned, uint32_t lane) {
    if (op == RO_SUM) {
        if constexpr (T == DT_BF16 || T == DT_FP16) {
            if (t.requant) {
                reduce_tile_tree<T, RO_SUM, true>(t, n, aligned, lane);
                return;
            }
        }
        reduce_tile_tree<T, RO_SUM, false>(t, n, aligned, lane);
    } else if (op == RO_MAX) {
        reduce_tile_tree<T, RO_MAX, false>(t, n, aligned, lane);
    } else {
        reduce_tile_tree<T, RO_MIN, false>(t, n, aligned, lane);
    }
}

__device__ __forceinline__ void run_reduce(uint32_t sig, uint32_t op, const TileOps& t, uint32_t n, bool aligned, uint32_t lane) {
    if (t.fold == FOLD_PAIRWISE) {
        switch (sig) {
            case SIG_BF16: run_tree<DT_BF16>(op, t, n, aligned, lane); break;
            case SIG_FP16: run_tree<DT_FP16>(op, t, n, aligned, lane); break;
            case SIG_FP32: run_tree<DT_FP32>(op, t, n, aligned, lane); break;
            case SIG_INT32: run_tree<DT_INT32>(op, t, n, aligned, lane); break;
            default: break;
        }
        return;
    }
    if (t.requant && op == RO_SUM) {
        // re-quantised partials only matter for 16-bit destinations
        if (sig == SIG_BF16) {
            reduce_tile<DT_BF16, DT_BF16, DT_BF16, RO_SUM, true>(t, n, aligned, lane);
            return;
        }
        if (sig == SIG_FP16) {
            reduce_tile<DT_FP16, DT_FP16, DT_FP16, RO_SUM, true>(t, n, aligned, lane);
            return;
        }
    }
    switch (sig) {
        case SIG_BF16: reduce_dispatch_op<DT_BF16, DT_BF16, DT_BF16>(op, t, n, aligned, lane); break;
        case SIG_FP16: reduce_dispatch_op<DT_FP16, DT_FP16, DT_FP16>(op, t, n, aligned, lane); break;
        case SIG_FP32: reduce_dispatch_op<DT_FP32, DT_FP32, DT_FP32>(op, t, n, aligned, lane); break;
        case SIG_INT32: reduce_dispatch_op<DT_INT32, DT_INT32, DT_INT32>(op, t, n, aligned, lane); break;
        case SIG_BF16_TO_F32: reduce_dispatch_op<DT_BF16, DT_BF16, DT_FP32>(op, t, n, aligned, lane); break;
        case SIG_F32_BF16_TO_F32: reduce_dispatch_op<DT_FP32, DT_BF16, DT_FP32>(op, t, n, aligned, lane); break;
        case SIG_F32_BF16_TO_BF16: reduce_dispatch_op<DT_FP32, DT_BF16, DT_BF16>(op, t, n, aligned, lane); break;
        case SIG_F32_TO_BF16: reduce_dispatch_op<DT_FP32, DT_FP32, DT_BF16>(op, t, n, aligned, lane); break;
        case SIG_FP16_TO_F32: reduce_dispatch_op<DT_FP16, DT_FP16, DT_FP32>(op, t, n, aligned, lane); break;
        case SIG_F32_FP16_TO_F32: reduce_dispatch_op<DT_FP32, DT_FP16, DT_FP32>(op, t, n, aligned, lane); break;
        case SIG_F32_FP16_TO_FP16: reduce_dispatch_op<DT_FP32, DT_FP16, DT_FP16>(op, t, n, aligned, lane); break;
        case SIG_F32_TO_FP16: reduce_dispatch_op<DT_FP32, DT_FP32, DT_FP16>(op, t, n, aligned, lane); break;
        default: break;
    }
}

// ------------------------------------------------------------------------------ COPY
// Byte copy of one source to every destination. 16-byte vectors when source and all
// destinations share their offset modulo 16 (a head and a tail of whole elements go one
// element per lane); element by element otherwise.
template <int ES>
__device__ __forceinline__ void copy_elems(const char* src, const TileOps& t, uint64_t first, uint64_t count, uint32_t lane) {
    typedef typename std::conditional<ES == 2, uint16_t, uint32_t>::type W;
    constexpr int U = 8;
    uint64_t e = first;
    for (; e + (uint64_t)U * kWaveSize <= first + count; e += (uint64_t)U * kWaveSize) {
        W v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = *gp<W>(src + (e + (uint64_t)u * kWaveSize + lane) * ES);
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d = (char*)from_lane(t.dst, j);
#pragma unroll
            for (int u = 0; u < U; ++u) *gp<W>(d + (e + (uint64_t)u * kWaveSize + lane) * ES) = v[u];
        }
    }
    for (uint64_t x = e + lane; x < first + count; x += kWaveSize) {
        W v = *gp<W>(src + x * ES);
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d = (char*)from_lane(t.dst, j);
            *gp<W>(d + x * ES) = v;
        }
    }
}

// Copy to destinations that share one offset modulo 16 that is not the source's (the int32 row
// ids of an AllToAllv, an AllGather of a count that is not a multiple of 16 bytes): after a head
// of fewer than 16 bytes every destination is 16-byte aligned, and every lane loads the 16 source
// bytes of its destination vector at the source's element alignment, one instruction instead of
// 16 / ES element loads (grouped AllToAllv of rows + ids 180.9-181.4 -> 179.6-180.0 us). A form
// that built each vector from two aligned loads and lane shuffles compiled to packed 32-bit
// moves, which the build rejects.
template <int ES>
__device__ __forceinline__ void copy_tile_shifted(const char* src, const TileOps& t, uint32_t n, uint32_t lane) {
    const uint64_t nbytes = (uint64_t)n * ES;
    uint64_t head = (16u - (from_lane(t.dst, 0) & 15u)) & 15u;
    if (head > nbytes) head = nbytes;
    if (head) copy_elems<ES>(src, t, 0, head / ES, lane);
    const char* s1 = src + head;
    const uint64_t nvec = (nbytes - head) / 16;
    constexpr int U = HCCL_COPY_UNROLL;
    uint64_t v0 = 0;
    for (; v0 + (uint64_t)U * kWaveSize <= nvec; v0 += (uint64_t)U * kWaveSize) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = vld_shifted<ES>(s1 + 16 * (v0 + (uint64_t)u * kWaveSize + lane));
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d1 = (char*)from_lane(t.dst, j) + head;
#pragma unroll
            for (int u = 0; u < U; ++u) vst_copy(d1 + 16 * (v0 + (uint64_t)u * kWaveSize + lane), v[u]);
        }
    }
    for (uint64_t v = v0 + lane; v < nvec; v += kWaveSize) {
        const u32x4 x = vld_shifted<ES>(s1 + 16 * v);
        for (uint32_t j = 0; j < t.ndst; ++j) vst_copy((char*)from_lane(t.dst, j) + head + 16 * v, x);
    }
    const uint64_t done = head + nvec * 16;
    if (done < nbytes) copy_elems<ES>(src, t, done / ES, (nbytes - done) / ES, lane);
}

template <int ES>
__device__ __forceinline__ void copy_tile(const TileOps& t, uint32_t n, uint32_t lane) {
    const char* src = (const char*)from_lane(t.src, 0);
    const uint32_t mis = (uint32_t)((uint64_t)src & 15u);
    // every destination must share the source's offset modulo 16 for the vector path
    const bool congruent =
        __ballot(lane < t.ndst && (uint32_t)(t.dst & 15u) != mis) == 0ull;
    if (!congruent) {
        // Destinations that agree among themselves modulo 16 still store whole vectors, except
        // 4-byte elements to several destinations: there element loads kept pace (all-gather of
        // 8 x (4 MiB + 4 B) int32 60 us element-wise, 73 us shifted; of 8 x (512 KiB + 2 B) bf16
        // 22.7 -> 13.5 us shifted).
        const uint32_t dmis = (uint32_t)(from_lane(t.dst, 0) & 15u);
        const bool agree = __ballot(lane < t.ndst && (uint32_t)(t.dst & 15u) != dmis) == 0ull;
        if (agree && (ES == 2 || t.ndst == 1)) copy_tile_shifted<ES>(src, t, n, lane);
        else copy_elems<ES>(src, t, 0, n, lane);
        return;
    }
    const uint64_t nbytes = (uint64_t)n * ES;
    uint64_t head = mis ? (16u - mis) : 0u;   // bytes before the first 16-byte boundary
    if (head > nbytes) head = nbytes;
    if (head) copy_elems<ES>(src, t, 0, head / ES, lane);
    constexpr int U = HCCL_COPY_UNROLL;
    constexpr uint64_t kStep = (uint64_t)U * kWaveSize * 16;
    uint64_t off = head;
    for (; off + kStep <= nbytes; off += kStep) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = vld(src + off + ((uint64_t)u * kWaveSize + lane) * 16);
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d = (char*)from_lane(t.dst, j);
#pragma unroll
            for (int u = 0; u < U; ++u) vst_copy(d + off + ((uint64_t)u * kWaveSize + lane) * 16, v[u]);
        }
    }
    for (; off + 16 * kWaveSize <= nbytes; off += 16 * kWaveSize) {
        u32x4 v = vld(src + off + (uint64_t)lane * 16);
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d = (char*)from_lane(t.dst, j);
            vst_copy(d + off + (uint64_t)lane * 16, v);
        }
    }
    {
        uint64_t x = off + (uint64_t)lane * 16;
        if (x + 16 <= nbytes) {
            u32x4 v = vld(src + x);
            for (uint32_t j = 0; j < t.ndst; ++j) {
                char* d = (char*)from_lane(t.dst, j);
                vst_copy(d + x, v);
            }
        }
        off += (nbytes - off) / 16 * 16;
    }
    if (off < nbytes) copy_elems<ES>(src, t, off / ES, (nbytes - off) / ES, lane);
}

// Copy of a tile whose source and destinations are all 16-byte aligned, U vectors per lane per
// step: every destination receives U KiB in a row per step.
template <int ES, int U = HCCL_COPY_UNROLL>
__device__ __forceinline__ void copy_tile_aligned(const TileOps& t, uint32_t n, uint32_t lane) {
    const char* src = (const char*)from_lane(t.src, 0);
    const uint64_t nbytes = (uint64_t)n * ES;
    constexpr uint64_t kStep = (uint64_t)U * kWaveSize * 16;
    uint64_t off = 0;
    for (; off + kStep <= nbytes; off += kStep) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = vld(src + off + ((uint64_t)u * kWaveSize + lane) * 16);
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d = (char*)from_lane(t.dst, j);
#pragma unroll
            for (int u = 0; u < U; ++u) vst_copy(d + off + ((uint64_t)u * kWaveSize + lane) * 16, v[u]);
        }
    }
    for (uint64_t x = off + (uint64_t)lane * 16; x + 16 <= nbytes; x += 16 * kWaveSize) {
        u32x4 v = vld(src + x);
        for (uint32_t j = 0; j < t.ndst; ++j) {
            char* d = (char*)from_lane(t.dst, j);
            vst_copy(d + x, v);
        }
    }
    off = nbytes / 16 * 16;
    if (off < nbytes) copy_elems<ES>(src, t, off / ES, (nbytes - off) / ES, lane);
}

// ---------------------------------------------------------------------- dependencies
__device__ __forceinline__ uint32_t load_relaxed(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until every dependency of the tile is satisfied. Returns false if the watchdog
// fired here or another wavefront recorded an error.
__device__ __forceinline__ bool wait_deps(const Dep* deps, uint32_t ndep, uint32_t k, uint32_t* state, ErrorRecord* err,
                          uint64_t timeout, uint32_t desc, uint32_t tile) {
    for (uint32_t i = 0; i < ndep; ++i) {
        const uint32_t kind = uni(deps[i].kind);
        const uint32_t expected = uni(deps[i].expected);
        const uint32_t word = uni(deps[i].state) + (kind == DEP_TILE ? k : 0u);
        const uint32_t* w = state + word;
        if (load_relaxed(w) >= expected) continue;
        const uint64_t t0 = wall_clock64();
        while (load_relaxed(w) < expected) {
            if (load_relaxed(&err->code) != 0u) return false;
            if (wall_clock64() - t0 > timeout) {
                if (__lane_id() == 0) {
                    uint32_t zero = 0;
                    if (__hip_atomic_compare_exchange_strong(&err->code, &zero, 1u, __ATOMIC_RELAXED,
                                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                        __hip_atomic_store(&err->desc, desc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        __hip_atomic_store(&err->tile, tile, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
                return false;
            }
            __builtin_amdgcn_s_sleep(2);
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return true;
}

// ----------------------------------------------------------------------- the kernel
// What every tile of a launch shares.
struct Shared {
    uint32_t* state;
    ErrorRecord* error;
    uint64_t timeout;
};

// Kernel specialisations: a program whose reductions all share one plain signature with SUM
// runs on the kernel built for that signature (only that path is compiled in, so registers
// are allocated for it alone); copy-only programs, and everything else, have their own.
template <int KIND>
__device__ __forceinline__ void exec_tile(uint32_t op, uint32_t sig, uint32_t redop, uint32_t es, const TileOps& ops,
                                          uint32_t n, bool aligned, uint32_t lane) {
    if (op == OP_REDUCE) {
        if constexpr (KIND == kKindGeneric) {
            run_reduce(sig, redop, ops, n, aligned, lane);
        } else if constexpr (KIND == SIG_BF16) {
            reduce_tile<DT_BF16, DT_BF16, DT_BF16, RO_SUM>(ops, n, aligned, lane);
        } else if constexpr (KIND == SIG_FP16) {
            reduce_tile<DT_FP16, DT_FP16, DT_FP16, RO_SUM>(ops, n, aligned, lane);
        } else if constexpr (KIND == SIG_FP32) {
            reduce_tile<DT_FP32, DT_FP32, DT_FP32, RO_SUM>(ops, n, aligned, lane);
        } else if constexpr (KIND == SIG_INT32) {
            reduce_tile<DT_INT32, DT_INT32, DT_INT32, RO_SUM>(ops, n, aligned, lane);
        }
    } else if (op == OP_COPY) {
        if constexpr (KIND == kKindCopyAligned) {
            // A copy to many destinations writes each of them in longer runs: 8 KiB per step
            // instead of 4 (8 vectors per lane; the kernel keeps 8 waves per SIMD). The copy phase
            // of the two-level all-reduce of 64 ranks: 4 MiB per rank 102 -> 90 us, 8 MiB
            // 184 -> 175 us, 32 MiB 736-757 -> 731-745 us; the all-gather of 64 x 512 KiB
            // 395-398 -> 388-393 us. 16 vectors per lane gained about 1 % more and would cost the
            // kernel three of its eight waves per SIMD.
            if (ops.ndst >= kWideStoreDsts) {
                if (es == 2) copy_tile_aligned<2, 8>(ops, n, lane);
                else copy_tile_aligned<4, 8>(ops, n, lane);
            } else {
                if (es == 2) copy_tile_aligned<2>(ops, n, lane);
                else copy_tile_aligned<4>(ops, n, lane);
            }
        } else {
            if (es == 2) copy_tile<2>(ops, n, lane);
            else copy_tile<4>(ops, n, lane);
        }
    }
}

// ---------------------------------------------------------------- AllToAllvDynamic
// The layout of a device-resident AllToAllv (Section IV-B-2) is read from device memory when
// the program runs. Every copy slot plans the whole exchange from the count matrix by itself,
// row by row with lane d standing for destination d, so no slot waits for another and nothing
// is shared between wavefronts: pass 1 checks every range and counts the dynamic tiles J,
// pass 2 walks the rows again and moves the slot's tiles k, k + S, k + 2S, ... Dynamic tiles are
// numbered source-major, then destination, then tile within the pair (destination-major in the
// register-resident form for P <= 8, dyn_slot_small). Strided like the static
// dispatch of a launched program, the slots work on one window of neighbouring tiles at a time:
// the grouped 2^18-row exchange of 8 ranks took 214 us with a contiguous run of J/S tiles per
// slot (thousands of separate streams at once), 202 us strided (194 us as a static AllToAllv),
// measured with 8 192 slots on a grid the CUs hold at once.

// Inclusive prefix sum over the lanes of a wavefront.
__device__ __forceinline__ uint64_t wave_scan_incl(uint64_t v, uint32_t lane) {
#pragma unroll
    for (uint32_t d = 1; d < (uint32_t)kWaveSize; d <<= 1) {
        const uint64_t t = __shfl_up(v, d);
        if (lane >= d) v += t;
    }
    return v;
}

struct DynView {     // a DynA2A record loaded into scalar registers
    uint32_t P, es, send0, recv0, counts, sdispls, rdispls, recvcounts, slots;
    uint64_t row_elems, send_cap, recv_cap, tile_elems;
};

// The record at byte `off` of the program image, read through the constant address space
// (scalar loads; records are 8-byte aligned, so 4- and 8-byte fields).
__device__ __forceinline__ DynView load_dyn(const uint8_t* prog, uint64_t off) {
    DynView v;
    v.P = cld<uint32_t>(prog, off + offsetof(DynA2A, P));
    v.es = cld<uint32_t>(prog, off + offsetof(DynA2A, elem_bytes));
    v.send0 = cld<uint32_t>(prog, off + offsetof(DynA2A, send0));
    v.recv0 = cld<uint32_t>(prog, off + offsetof(DynA2A, recv0));
    v.counts = cld<uint32_t>(prog, off + offsetof(DynA2A, counts));
    v.sdispls = cld<uint32_t>(prog, off + offsetof(DynA2A, sdispls));
    v.rdispls = cld<uint32_t>(prog, off + offsetof(DynA2A, rdispls));
    v.recvcounts = cld<uint32_t>(prog, off + offsetof(DynA2A, recvcounts));
    v.slots = cld<uint32_t>(prog, off + offsetof(DynA2A, slots));
    v.row_elems = cld<uint64_t>(prog, off + offsetof(DynA2A, row_elems));
    v.send_cap = cld<uint64_t>(prog, off + offsetof(DynA2A, send_cap));
    v.recv_cap = cld<uint64_t>(prog, off + offsetof(DynA2A, recv_cap));
    v.tile_elems = cld<uint64_t>(prog, off + offsetof(DynA2A, tile_elems));
    return v;
}

// Slot k of an AllToAllvDynamic.
//  Pass 1, lane i standing for rank i: walks row i of the count matrix (what source i sends) and
//  column i (what destination i receives) with per-lane sums only, checks every range as the
//  oracle does (a packed side fits iff its total fits, since counts are non-negative), and
//  counts the dynamic tiles of row i. One scan over the lanes then gives each row's first tile.
//  Pass 2, lane d standing for destination d: from the row holding the slot's first tile, works
//  out the pairs' offsets and moves the slot's tiles.
// ES / ER: the exchange has explicit send / receive offsets.
template <int KIND, bool ES, bool ER>
__device__ __forceinline__ void dyn_slot(const DynView& a, uint32_t k, const uint64_t* bufs, ErrorRecord* err,
                                         uint32_t desc, uint32_t lane) {
    constexpr uint32_t B = 2;  // rows whose loads are in flight together
    const uint32_t P = a.P;
    const bool on = lane < P;
    const uint64_t R = a.row_elems, te = a.tile_elems;
    const int64_t* counts = (const int64_t*)uni64(bufs[a.counts]);
    const int64_t* sdis = ES ? (const int64_t*)uni64(bufs[a.sdispls]) : nullptr;
    const int64_t* rdis = ER ? (const int64_t*)uni64(bufs[a.rdispls]) : nullptr;
    const uint64_t cmax = a.send_cap < a.recv_cap ? a.send_cap : a.recv_cap;

    // ---- pass 1
    bool bad = false;
    uint64_t srow = 0, scol = 0, trow = 0;  // rows sent, rows received, tiles of row `lane`
    for (uint32_t t0 = 0; t0 < P; t0 += B) {
        int64_t cr[B], cc[B];
#pragma unroll
        for (uint32_t u = 0; u < B; ++u) {
            const bool in = on && t0 + u < P;
            cr[u] = in ? counts[(uint64_t)lane * P + t0 + u] : 0;  // source lane -> destination t
            cc[u] = in ? counts[(uint64_t)(t0 + u) * P + lane] : 0;  // source t -> destination lane
        }
#pragma unroll
        for (uint32_t u = 0; u < B; ++u) {
            const uint32_t t = t0 + u;
            if (t < P) {
                bad |= on && (cr[u] < 0 || (uint64_t)cr[u] > cmax);
                const uint64_t c = (cr[u] > 0 && (uint64_t)cr[u] <= cmax) ? (uint64_t)cr[u] : 0;
                const uint64_t c2 = (cc[u] > 0 && (uint64_t)cc[u] <= cmax) ? (uint64_t)cc[u] : 0;
                srow = (srow > ~0ull - c) ? ~0ull : srow + c;  // saturating: 64 counts near the
                scol = (scol > ~0ull - c2) ? ~0ull : scol + c2;  // capacity limit could wrap
                trow += (c * R + te - 1) / te;
                if constexpr (ES) {
                    const int64_t x = on ? sdis[(uint64_t)lane * P + t] : 0;
                    if (c && (x < 0 || (uint64_t)x > a.send_cap || c > a.send_cap - (uint64_t)x)) bad = true;
                }
                if constexpr (ER) {
                    const int64_t x = on ? rdis[(uint64_t)lane * P + t] : 0;
                    if (c2 && (x < 0 || (uint64_t)x > a.recv_cap || c2 > a.recv_cap - (uint64_t)x)) bad = true;
                }
            }
        }
    }
    if (!ES && srow > a.send_cap) bad = true;
    if (!ER && scol > a.recv_cap) bad = true;
    if constexpr (ER) {
        // non-empty receive ranges of one destination must not overlap (lane = source here; a
        // range that is out of bounds has already failed, so only in-bounds sums are trusted)
        for (uint32_t d = 0; d < P; ++d) {
            const int64_t cx = on ? counts[(uint64_t)lane * P + d] : 0;
            const int64_t rx = on ? rdis[(uint64_t)d * P + lane] : 0;
            const uint64_t c = (cx > 0) ? (uint64_t)cx : 0, r = (uint64_t)rx;
            for (uint32_t j = 0; j < P; ++j) {
                const uint64_t cj = from_lane(c, j), rj = from_lane(r, j);
                if (j != lane && c && cj && r < rj + cj && rj < r + c) bad = true;
            }
        }
    }
    const bool rejected = __ballot(bad) != 0ull;
    if (k == 0) {
        // slot 0 reports: the received counts, always, and a rejected layout
        if (a.recvcounts != kNoBuffer) {
            int64_t* rc = (int64_t*)uni64(bufs[a.recvcounts]);
            for (uint32_t t = 0; t < P; ++t)
                if (on) rc[(uint64_t)lane * P + t] = counts[(uint64_t)t * P + lane];
        }
        if (rejected && lane == 0) {
            uint32_t zero = 0;
            if (__hip_atomic_compare_exchange_strong(&err->code, &zero, 2u, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT)) {
                __hip_atomic_store(&err->desc, desc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&err->tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
    if (rejected) return;  // move nothing

    // ---- pass 2
    const uint64_t gincl = wave_scan_incl(trow, lane);  // lane s: tiles of rows 0..s
    const uint64_t J = from_lane(gincl, P - 1);
    const uint64_t S = a.slots;
    if (k >= J) return;
    // the row holding tile k (rows with no tiles before it are skipped by the ballot)
    uint32_t s = (uint32_t)__popcll(__ballot(on && gincl <= k));
    uint64_t G = s ? from_lane(gincl, s - 1) : 0;  // tiles of the rows before s
    // lane d: rows destination d receives from the sources before s (the packed receive offset)
    uint64_t col = 0;
    if constexpr (!ER) {
        for (uint32_t q0 = 0; q0 < s; q0 += B) {
            int64_t cq[B];
#pragma unroll
            for (uint32_t u = 0; u < B; ++u) cq[u] = (on && q0 + u < s) ? counts[(uint64_t)(q0 + u) * P + lane] : 0;
#pragma unroll
            for (uint32_t u = 0; u < B; ++u) col += (uint64_t)cq[u];
        }
    }
    TileOps ops;
    ops.nsrc = 1;
    ops.ndst = 1;
    ops.group = 0;
    const uint64_t send_elems = a.send_cap * R, recv_elems = a.recv_cap * R;
    for (; s < P && G < J; ++s) {
        // checked in pass 1; clamped again so that a count rewritten while this runs (a race in
        // the caller) still cannot move a byte outside the buffers (see the guard below)
        const int64_t cx = on ? counts[(uint64_t)s * P + lane] : 0;
        const uint64_t c = (cx > 0 && (uint64_t)cx <= cmax) ? (uint64_t)cx : 0;
        uint64_t so, ro;
        if constexpr (ES) so = on ? (uint64_t)sdis[(uint64_t)s * P + lane] : 0;
        else so = wave_scan_incl(c, lane) - c;
        if constexpr (ER) {
            ro = on ? (uint64_t)rdis[(uint64_t)lane * P + s] : 0;
        } else {
            ro = col;
            col += c;
        }
        const uint64_t ne = c * R;
        const uint64_t pre = wave_scan_incl((ne + te - 1) / te, lane);
        const uint64_t T = from_lane(pre, P - 1);
        // this slot's tiles of the row: k, k + S, k + 2S, ... from G on
        const uint64_t lo = (G <= k) ? k : k + (G - k + S - 1) / S * S, hi = G + T;
        const uint64_t src_base = uni64(bufs[a.send0 + s]);
        for (uint64_t j = lo; j < hi; j += S) {
            const uint64_t jr = j - G;  // < T, so the destination below is < P
            const uint32_t d = (uint32_t)__popcll(__ballot(on && pre <= jr));
            if (d >= P) break;
            const uint64_t t = jr - (d ? from_lane(pre, d - 1) : 0);
            const uint64_t e0 = t * te, n_pair = from_lane(ne, d);
            const uint32_t n = (uint32_t)((n_pair - e0 < te) ? (n_pair - e0) : te);
            const uint64_t sod = from_lane(so, d), rod = from_lane(ro, d);
            if (sod > a.send_cap || rod > a.recv_cap || sod * R + e0 + n > send_elems ||
                rod * R + e0 + n > recv_elems)
                continue;  // only a caller race on the metadata gets here
            ops.src = src_base + (sod * R + e0) * a.es;
            ops.dst = uni64(bufs[a.recv0 + d]) + (rod * R + e0) * a.es;
            exec_tile<KIND>(OP_COPY, 0, 0, a.es, ops, n, false, lane);
        }
        G += T;
    }
}

// Slot k of an AllToAllvDynamic with P*P <= 64 (P <= 8): lane l stands for the pair
// (s, d) = (l % P, l / P), so one load brings the whole count matrix into registers; row and
// column sums, the packed offsets and the overlap checks are P shuffles each, and the tiles
// are found with one scan, with no further loads. Same rules and results as dyn_slot; the
// dynamic tiles are numbered destination-major here (the slots then fill one receive buffer at
// a time, as the static exchange does: headline exchange 189.6-192.4 -> 189.4-190.8 us).
template <int KIND, bool ES, bool ER>
__device__ __forceinline__ void dyn_slot_small(const DynView& a, uint32_t k, const uint64_t* bufs, ErrorRecord* err,
                                               uint32_t desc, uint32_t lane) {
    const uint32_t P = a.P, PP = a.P * a.P;
    const bool on = lane < PP;
    const uint32_t s = on ? lane % P : 0u, d = on ? lane / P : 0u;
    const uint64_t R = a.row_elems, te = a.tile_elems;
    const uint64_t cmax = a.send_cap < a.recv_cap ? a.send_cap : a.recv_cap;
    const int64_t* counts = (const int64_t*)uni64(bufs[a.counts]);
    const int64_t cx = on ? counts[(uint64_t)s * P + d] : 0;
    bool bad = on && (cx < 0 || (uint64_t)cx > cmax);
    const uint64_t c = (on && !bad) ? (uint64_t)cx : 0;  // at most 2^59: sums of 8 cannot wrap
    uint64_t row = 0, col = 0, row_before = 0, col_before = 0;
    for (uint32_t j = 0; j < P; ++j) {
        const uint64_t cr = __shfl(c, (int)(j * P + s));  // pair (s, j)
        const uint64_t cc = __shfl(c, (int)(d * P + j));  // pair (j, d)
        row += cr;
        col += cc;
        if (j < d) row_before += cr;
        if (j < s) col_before += cc;
    }
    uint64_t so, ro;
    if constexpr (ES) {
        const int64_t x = on ? ((const int64_t*)uni64(bufs[a.sdispls]))[(uint64_t)s * P + d] : 0;
        if (c && (x < 0 || (uint64_t)x > a.send_cap || c > a.send_cap - (uint64_t)x)) bad = true;
        so = (uint64_t)x;
    } else {
        if (on && row > a.send_cap) bad = true;  // a packed source fits iff its total fits
        so = row_before;
    }
    if constexpr (ER) {
        const int64_t x = on ? ((const int64_t*)uni64(bufs[a.rdispls]))[(uint64_t)d * P + s] : 0;
        if (c && (x < 0 || (uint64_t)x > a.recv_cap || c > a.recv_cap - (uint64_t)x)) bad = true;
        ro = (uint64_t)x;
        // the other sources of destination d (an out-of-bounds range has already failed)
        for (uint32_t j = 0; j < P; ++j) {
            const uint64_t cj = __shfl(c, (int)(d * P + j)), rj = __shfl(ro, (int)(d * P + j));
            if (j != s && c && cj && ro < rj + cj && rj < ro + c) bad = true;
        }
    } else {
        if (on && col > a.recv_cap) bad = true;
        ro = col_before;
    }
    const bool rejected = __ballot(bad) != 0ull;
    if (k == 0) {
        if (a.recvcounts != kNoBuffer && on) ((int64_t*)uni64(bufs[a.recvcounts]))[(uint64_t)d * P + s] = cx;
        if (rejected && lane == 0) {
            uint32_t zero = 0;
            if (__hip_atomic_compare_exchange_strong(&err->code, &zero, 2u, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT)) {
                __hip_atomic_store(&err->desc, desc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&err->tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
    if (rejected) return;  // move nothing

    const uint64_t ne = c * R;
    const uint64_t incl = wave_scan_incl((ne + te - 1) / te, lane);  // tiles of pairs 0..l
    const uint64_t J = from_lane(incl, kWaveSize - 1);
    const uint64_t send_elems = a.send_cap * R, recv_elems = a.recv_cap * R;
    TileOps ops;
    ops.nsrc = 1;
    ops.ndst = 1;
    ops.group = 0;
    for (uint64_t j = k; j < J; j += a.slots) {
        const uint32_t pr = (uint32_t)__popcll(__ballot(incl <= j));  // j < J, so pr < P*P
        if (pr >= PP) break;
        const uint64_t t = j - (pr ? from_lane(incl, pr - 1) : 0);
        const uint64_t e0 = t * te, n_pair = from_lane(ne, pr);
        const uint32_t n = (uint32_t)((n_pair - e0 < te) ? (n_pair - e0) : te);
        const uint64_t sod = from_lane(so, pr), rod = from_lane(ro, pr);
        if (sod > a.send_cap || rod > a.recv_cap || sod * R + e0 + n > send_elems || rod * R + e0 + n > recv_elems)
            continue;  // only a caller race on the metadata gets here
        ops.src = uni64(bufs[a.send0 + pr % P]) + (sod * R + e0) * a.es;
        ops.dst = uni64(bufs[a.recv0 + pr / P]) + (rod * R + e0) * a.es;
        exec_tile<KIND>(OP_COPY, 0, 0, a.es, ops, n, false, lane);
    }
}

template <int KIND>
__device__ __forceinline__ bool run_tile(const Shared& a, const uint8_t* prog, const ProgramHeader& h, uint32_t t,
                                         uint32_t lane, const uint64_t* bufs, bool stamp, uint64_t& ready) {
    const uint32_t d = uni(((const uint32_t*)(prog + h.off_tile_desc))[t]);
    // The descriptor arrives as four 16-byte scalar loads through the constant address space
    // (its fields sit in the words named below). Against per-field vector loads: the two-level
    // all-reduce of 64 ranks and the reduce-scatter P=8 x 256 MiB -1 %, AllToAllvDynamic -1 %,
    // the ring all-reduce P=4 x 2^20 fp32 -2 %, the grouped AllToAllv -0.5 %; a 1 GiB copy of 1 024
    // one-chunk steps +3 %. The tile table itself (one word per tile, up to megabytes) stays on
    // the vector path: through the scalar cache it cost that copy 4 % and gained nothing else.
    const uint64_t Db = h.off_desc + (uint64_t)sizeof(Desc) * d;
    const u32x4 w0 = cld<u32x4>(prog, Db);       // op redop flags sig | nsrc ndst | group ndep | src
    const u32x4 w1 = cld<u32x4>(prog, Db + 16);  // dst | dep | tile0 | ntiles
    const u32x4 w2 = cld<u32x4>(prog, Db + 32);  // tile_elems | - | nelem
    const u32x4 w3 = cld<u32x4>(prog, Db + 48);  // fold | requant | aux | -
    const uint32_t op = w0[0] & 0xFFu;
    const uint32_t flags = (w0[0] >> 16) & 0xFFu;
    const uint32_t ndep = w0[2] >> 16;
    const uint32_t k = t - w1[2];
    const uint64_t te = w2[0];
    const uint64_t nelem = (uint64_t)w2[2] | ((uint64_t)w2[3] << 32);
    const uint64_t e0 = (uint64_t)k * te;
    const uint32_t n = (uint32_t)((nelem - e0 < te) ? (nelem - e0) : te);

    if (ndep) {
        const Dep* deps = (const Dep*)(prog + h.off_dep) + w1[1];
        if (!wait_deps(deps, ndep, k, a.state, a.error, a.timeout, d, t)) return false;
    }
    if (stamp) ready = wall_clock64();

    if (op == OP_DYN_COPY) {
        // the host runs programs with dynamic steps on these two kernels only
        if constexpr (KIND == kKindDynamic || KIND == kKindGeneric) {
            const DynView v = load_dyn(prog, h.off_aux + (uint64_t)sizeof(DynA2A) * w3[2]);
            const bool es = v.sdispls != kNoBuffer, er = v.rdispls != kNoBuffer;
            // the register-resident planner only in the dynamic kernel: the generic one carries
            // every other path already, and the general planner covers every P
            bool small = false;
            if constexpr (KIND == kKindDynamic) {
                small = v.P * v.P <= (uint32_t)kWaveSize;
                if (small) {
                    if (!es && !er) dyn_slot_small<KIND, false, false>(v, k, bufs, a.error, d, lane);
                    else if (es && !er) dyn_slot_small<KIND, true, false>(v, k, bufs, a.error, d, lane);
                    else if (!es) dyn_slot_small<KIND, false, true>(v, k, bufs, a.error, d, lane);
                    else dyn_slot_small<KIND, true, true>(v, k, bufs, a.error, d, lane);
                }
            }
            if (!small) {
                if (!es && !er) dyn_slot<KIND, false, false>(v, k, bufs, a.error, d, lane);
                else if (es && !er) dyn_slot<KIND, true, false>(v, k, bufs, a.error, d, lane);
                else if (!es) dyn_slot<KIND, false, true>(v, k, bufs, a.error, d, lane);
                else dyn_slot<KIND, true, true>(v, k, bufs, a.error, d, lane);
            }
        }
    } else {
        TileOps ops;
        ops.nsrc = w0[1] & 0xFFFFu;
        ops.ndst = w0[1] >> 16;
        ops.group = w0[2] & 0xFFFFu;
        ops.fold = w3[0];
        ops.requant = w3[1];
        const Operand* opl = (const Operand*)(prog + h.off_operand);
        ops.src = 0;
        ops.dst = 0;
        bool misaligned = false;
        if (lane < ops.nsrc) {
            Operand o = opl[w0[3] + lane];
            ops.src = bufs[o.buf] + o.offset + e0 * elem_bytes(o.dtype);
            misaligned |= (ops.src & 15u) != 0;
        }
        if (lane < ops.ndst) {
            Operand o = opl[w1[0] + lane];
            ops.dst = bufs[o.buf] + o.offset + e0 * elem_bytes(o.dtype);
            misaligned |= (ops.dst & 15u) != 0;
        }
        const uint32_t es0 = elem_bytes(cld<uint32_t>(prog, h.off_operand + 16ull * w0[3] + 4));
        exec_tile<KIND>(op, w0[0] >> 24, (w0[0] >> 8) & 0xFFu, es0, ops, n, __ballot(misaligned) == 0ull, lane);
    }

    if (flags) {
        // make this tile's stores visible device-wide before the signal
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        if (lane == 0) {
            if (flags & DF_SIGNAL_DESC)
                __hip_atomic_fetch_add(a.state + kStateDescBase + d, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (flags & DF_SIGNAL_TILE)
                __hip_atomic_store(a.state + kStateDescBase + h.ndesc + t, 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    return true;
}

// Runs tile t and, when the launch is traced, records its times and place (lane 0 writes).
// Only the generic kernel carries the trace code (the host runs traced launches on it): the
// clock reads and the record stores in the tile loop of the specialised kernels, even when
// skipped, measured 8 % slower copies.
template <int KIND>
__device__ __forceinline__ bool run_tile_traced(const Shared& a, const uint8_t* prog, const ProgramHeader& h,
                                                uint32_t t, uint32_t lane, const uint64_t* bufs, TileStamp* trace,
                                                uint32_t wave) {
    if constexpr (KIND != kKindGeneric) {
        uint64_t unused = 0;
        return run_tile<KIND>(a, prog, h, t, lane, bufs, false, unused);
    }
    // one inlined copy of the tile code whether or not the launch is traced
    const uint64_t t0 = trace ? wall_clock64() : 0;
    uint64_t ready = t0;
    const bool ok = run_tile<KIND>(a, prog, h, t, lane, bufs, trace != nullptr, ready);
    if (trace && lane == 0) {
        const uint64_t t2 = wall_clock64();
        // HW_ID: SIMD [5:4], CU [11:8], shader engine [15:13]; XCC_ID [3:0]
        const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);
        const uint32_t xcc = __builtin_amdgcn_s_getreg((15 << 11) | 20) & 0xFu;
        // two 16-byte stores straight from registers (a TileStamp temporary would live in scratch)
        u32x4 lo, hi;
        lo[0] = (uint32_t)t0;
        lo[1] = (uint32_t)(t0 >> 32);
        lo[2] = (uint32_t)(ready - t0);
        lo[3] = (uint32_t)(t2 - t0);
        hi[0] = wave;
        hi[1] = (xcc << 24) | (((hw >> 13) & 7u) << 16) | (((hw >> 8) & 0xFu) << 8) | ((hw >> 4) & 3u);
        hi[2] = 0;
        hi[3] = 0;
        u32x4* rec = (u32x4*)(trace + t);
        rec[0] = lo;
        rec[1] = hi;
    }
    return ok;
}

// ------------------------------------------------------------------ device trigger
// A pre-launched collective holds until a device word satisfies a comparison (Section IV-B-3:
// the caller attaches an address and a comparator; the collective is enqueued at once and
// blocks on the device until the compute side signals). One thread per workgroup polls the
// word with system-scope loads (the writer may be another kernel, a copy or the host), backing
// off between polls up to about a microsecond so that a long wait does not load the memory
// channel that holds the word; the rest of the workgroup waits at the barrier, issuing no
// memory traffic. Returns false when the watchdog fired or another workgroup recorded an error.
__device__ __forceinline__ bool trigger_cmp(uint64_t x, uint64_t v, uint32_t cmp) {
    switch (cmp) {
        case CMP_EQ: return x == v;
        case CMP_NE: return x != v;
        case CMP_GE: return x >= v;
        case CMP_GT: return x > v;
        case CMP_LE: return x <= v;
        default: return x < v;
    }
}

__device__ __forceinline__ bool trigger_wait(const LaunchArgs& a) {
    __shared__ uint32_t go;
    if (threadIdx.x == 0) {
        uint32_t ok = 1, nap = 1;
        const uint64_t t0 = wall_clock64();
        while (!trigger_cmp(__hip_atomic_load(a.wait_addr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM),
                            a.wait_value, a.wait_cmp)) {
            if (load_relaxed(&a.error->code) != 0u) {
                ok = 0;
                break;
            }
            if (wall_clock64() - t0 > a.timeout_ticks) {
                uint32_t zero = 0;
                if (__hip_atomic_compare_exchange_strong(&a.error->code, &zero, 3u, __ATOMIC_RELAXED,
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                    __hip_atomic_store(&a.error->tile, blockIdx.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ok = 0;
                break;
            }
            // s_sleep takes a constant: 64 x (1, 2, 4, ..., 32) clocks
            if (nap == 1) __builtin_amdgcn_s_sleep(1);
            else if (nap == 2) __builtin_amdgcn_s_sleep(2);
            else if (nap == 4) __builtin_amdgcn_s_sleep(4);
            else if (nap == 8) __builtin_amdgcn_s_sleep(8);
            else if (nap == 16) __builtin_amdgcn_s_sleep(16);
            else __builtin_amdgcn_s_sleep(32);
            if (nap < 32) nap *= 2;
        }
        // whatever the signalling side wrote before the word is visible from here on
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        go = ok;
    }
    __syncthreads();
    return go != 0u;
}

// At least four waves per SIMD for the specialised kernels, five for the 16-bit SUM reductions
// (they fit in 96 VGPRs without spilling: the reduce-scatter P=8 x 256 MiB bf16 confined to 16
// CUs, where few wavefronts carry every tile, 2.85 -> 2.70 ms; on the whole chip no change);
// the generic kernel (every fold, mixed types) may use more registers rather than spill.
template <int KIND>
constexpr int kMinWavesPerEu = KIND == kKindGeneric ? 3 : (KIND == SIG_BF16 || KIND == SIG_FP16) ? 5 : 4;

template <int KIND>
__global__ void __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(kMinWavesPerEu<KIND>)))
hccl_executor(LaunchArgs a) {
    const uint32_t lane = __lane_id();
    // The hardware deals workgroups to the XCDs in turn (block b to XCD b mod 8). With xcd_order
    // the blocks of one XCD take consecutive numbers, so at any moment each XCD (its L2 and its
    // address-translation caches) works on one contiguous stretch of the tiles.
    uint32_t block = blockIdx.x;
    if (a.xcd_order) {
        const uint32_t B = gridDim.x, x = block % kXcds, j = block / kXcds;
        block = x * (B / kXcds) + (x < B % kXcds ? x : B % kXcds) + j;
    }
    const uint32_t wave = uni(block * kWavesPerBlock + (threadIdx.x / kWaveSize));
    const uint8_t* prog = a.prog;
    ProgramHeader h;
    h.ndesc = cld<uint32_t>(prog, offsetof(ProgramHeader, ndesc));
    h.ntiles = cld<uint32_t>(prog, offsetof(ProgramHeader, ntiles));
    h.nstate = cld<uint32_t>(prog, offsetof(ProgramHeader, nstate));
    h.off_desc = cld<uint64_t>(prog, offsetof(ProgramHeader, off_desc));
    h.off_operand = cld<uint64_t>(prog, offsetof(ProgramHeader, off_operand));
    h.off_dep = cld<uint64_t>(prog, offsetof(ProgramHeader, off_dep));
    h.off_tile_desc = cld<uint64_t>(prog, offsetof(ProgramHeader, off_tile_desc));
    h.off_aux = cld<uint64_t>(prog, offsetof(ProgramHeader, off_aux));
    // the buffer table is indexed per lane, so it is read from the kernel-argument segment
    const uint64_t* bufs = (const uint64_t*)((const char*)__builtin_amdgcn_kernarg_segment_ptr() +
                                             offsetof(LaunchArgs, bufs));

    Shared sh;
    sh.state = a.state;
    sh.error = a.error;
    sh.timeout = a.timeout_ticks;
    const uint32_t nworkers = a.nworkers;

    const bool has_deps = (cld<uint32_t>(prog, offsetof(ProgramHeader, flags)) & PF_HAS_DEPS) != 0u;
    const bool triggered = a.wait_addr != nullptr;
    // a workgroup whose trigger wait failed runs no tile but still counts itself done below
    const bool started = !triggered || trigger_wait(a);
    // this launch runs one phase of the program: tiles [tile_begin, tile_end)
    const uint32_t tb = a.tile_begin, te = a.tile_end;
    if (started && !a.dynamic) {
        // Wavefront w runs tiles w, w + W, w + 2W, ... of the phase in order (only tile w when
        // the host gave the launch one wavefront per tile, as it does when no tile waits). Without
        // dependencies no tile waits for another, so any residency drains. A dependent program
        // needs the whole grid resident (the host then sizes it to the CUs the stream may use and
        // sends it here only while no waiting executor holds CUs): a tile waits only for lower
        // tiles, everything a wavefront ran before is lower, and the lowest unfinished tile is
        // always running.
        for (uint32_t t = tb + wave; t < te; t += nworkers) {
            if ((has_deps || triggered) && load_relaxed(&a.error->code) != 0u) break;
            if (!run_tile_traced<KIND>(sh, prog, h, t, lane, bufs, a.trace, wave)) break;
        }
    } else if (started) {
        // Tiles by ticket, in program order: a tile is only ever held by a running wavefront,
        // and it waits only for lower tiles, which running wavefronts took before it; so the
        // program drains whatever part of the grid is resident (a resident or a triggered
        // executor may hold CUs). The first tiles are taken per workgroup, one atomic for its
        // four wavefronts (the start is when every wavefront would hit the counter).
        uint32_t* ticket = a.state + kStateTicket;
        __shared__ uint32_t first;
        if (threadIdx.x == 0)
            first = __hip_atomic_fetch_add(ticket, (uint32_t)kWavesPerBlock, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        uint32_t t = uni(tb + first + threadIdx.x / kWaveSize);
        // with at least as many wavefronts as tiles the first tickets cover every tile
        const bool more = te - tb > nworkers;
        while (t < te) {
            if (load_relaxed(&a.error->code) != 0u) break;
            // claim the next ticket now; its latency hides behind this tile's work
            uint32_t next = te;
            if (more && lane == 0)
                next = tb + __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (!run_tile_traced<KIND>(sh, prog, h, t, lane, bufs, a.trace, wave)) break;
            t = uni(__shfl(next, 0));
        }
    }

    // no counter was touched (the same for every thread of the grid)
    if (!has_deps && !a.dynamic) return;

    // The last workgroup to finish clears the counters for the next launch (one atomic per
    // workgroup: same-address atomics from thousands of wavefronts would serialise). Every
    // counter update is an agent-scope atomic, so it is enough that each wavefront's updates
    // have completed (vmcnt(0) counts stores and atomics on this GPU) before its workgroup
    // counts itself done.
    __shared__ uint32_t last_block;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev =
            __hip_atomic_fetch_add(a.state + kStateDone, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last_block = (prev == gridDim.x - 1) ? 1u : 0u;
    }
    __syncthreads();
    if (last_block) {
        for (uint32_t i = threadIdx.x; i < h.nstate; i += kBlockThreads)
            __hip_atomic_store(a.state + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The completion word of a triggered collective, launched right behind the executor on its
// stream (the paper's dedicated subgraph for the set, Section IV-B-3): the executor's results
// are visible device-wide once it has ended, which costs nothing extra, whereas a write-back
// of the L2 by every workgroup before a word set from inside the executor measured 15-20 us.
// Nothing is written if the launch recorded an error.
__global__ void hccl_signal(uint64_t* word, uint64_t value, const ErrorRecord* err) {
    if (threadIdx.x == 0 && blockIdx.x == 0 &&
        __hip_atomic_load(&err->code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u)
        __hip_atomic_store(word, value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// ------------------------------------------------------------------ resident executor
// An executor that stays running and takes work packets through a doorbell in host memory
// (Section II-A-2: the message engine's control core waits for work and unrolls each packet as
// it arrives; Section V-B: re-enqueueing a cached packet is the whole per-call cost). The host
// writes a packet's arguments into a ring slot, then its sequence number. The last workgroup
// is the relay: its thread 0 polls that number with system-scope loads, the workgroup copies
// the arguments into a device mirror and publishes the number in device memory, so that only
// one workgroup pays the PCIe round trips. Every workgroup then copies the arguments into LDS
// and runs its share of the tiles exactly as a launched executor does (wavefront w takes tiles
// w, w + W, ...). The last workgroup to finish clears the program's counters, writes the
// results back for readers outside the GPU and stores the sequence number in host memory; the
// relay waits for that before it publishes the next packet, and fetches that packet meanwhile
// if it has arrived. Every wait is bounded: the relay ends the executor after `idle_ticks`
// without a packet, and a workgroup that waits longer than its limit for the others ends too.
__device__ __forceinline__ void backoff(uint32_t& nap, uint32_t cap) {
    if (nap == 1) __builtin_amdgcn_s_sleep(1);
    else if (nap == 2) __builtin_amdgcn_s_sleep(2);
    else if (nap == 4) __builtin_amdgcn_s_sleep(4);
    else if (nap == 8) __builtin_amdgcn_s_sleep(8);
    else if (nap == 16) __builtin_amdgcn_s_sleep(16);
    else __builtin_amdgcn_s_sleep(32);
    if (nap < cap) nap *= 2;
}

// Polls a device word until it equals `want`; false after `limit` wall-clock ticks.
__device__ __forceinline__ bool wait_word(const uint32_t* w, uint32_t want, uint64_t limit) {
    uint32_t nap = 1;
    const uint64_t t0 = wall_clock64();
    while (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want) {
        if (wall_clock64() - t0 > limit) return false;
        backoff(nap, 4);
    }
    return true;
}

__global__ void __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(3)))
hccl_resident(ResidentArgs r) {
    static_assert(sizeof(LaunchArgs) % 8 == 0, "the packet is copied in 8-byte words");
    constexpr uint32_t kWords = sizeof(LaunchArgs) / 8;
    __shared__ uint64_t pk[kWords];
    __shared__ uint32_t stop;
    __shared__ uint32_t last_block;
    __shared__ uint32_t ahead;       // relay: the next packet is already in pk and its mirror
    __shared__ uint32_t ahead_stop;  // relay: ... and it is the stop request
    __shared__ uint32_t sig, fetch;  // relay: decisions of thread 0 while it waits
    __shared__ uint32_t why;         // relay: why it stopped (ResidentExit)
    const uint32_t lane = __lane_id();
    const uint32_t wave = uni(blockIdx.x * kWavesPerBlock + (threadIdx.x / kWaveSize));
    const uint32_t nworkers = gridDim.x * kWavesPerBlock;
    // the relay is the last workgroup: its wavefronts come last in the tile order, so on small
    // packets it has no tiles and is free to fetch the next packet while the others work
    const bool relay = blockIdx.x == gridDim.x - 1;
    uint32_t* const arrived = r.ctl;
    uint32_t* const finished = r.ctl + 1;
    uint32_t* const published = r.ctl + 2;
    uint32_t* const stop_flag = r.ctl + 3;
    if (threadIdx.x == 0) {
        ahead = 0;
        ahead_stop = 0;
        why = RESIDENT_EXIT_STOP;
    }
    __syncthreads();

    for (uint64_t k = 1;; ++k) {
        uint64_t* const mirror = r.mirror + (k & 1) * kWords;  // two copies: one is filled ahead
        if (relay) {
            ResidentSlot* slot = &r.q->slots[(k - 1) % kResidentSlots];
            if (threadIdx.x == 0) {
                uint32_t end = 0;
                if (ahead) {
                    end = ahead_stop;
                } else {
                    uint32_t nap = 1;
                    const uint64_t t0 = wall_clock64();
                    for (;;) {
                        const uint64_t v = __hip_atomic_load(&slot->seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                        if ((v & ~kResidentStop) == k) {
                            end = (v & kResidentStop) ? 1u : 0u;
                            break;
                        }
                        if (wall_clock64() - t0 > r.idle_ticks) {
                            end = 1;
                            why = RESIDENT_EXIT_IDLE;
                            break;
                        }
                        backoff(nap, 4);
                    }
                    // the slot's arguments, and whatever was written to the packet's buffers
                    // before the doorbell, are visible from here on (stale lines are dropped)
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
                }
                stop = end;
            }
            __syncthreads();
            if (!stop && !ahead) {
                const uint64_t* from = (const uint64_t*)&slot->args;
                for (uint32_t i = threadIdx.x; i < kWords; i += kBlockThreads) {
                    const uint64_t w = __hip_atomic_load(from + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                    pk[i] = w;
                    __hip_atomic_store(mirror + i, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (threadIdx.x == 0) {
                ahead = 0;
                __hip_atomic_store(stop_flag, stop, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(published, (uint32_t)k, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            }
        } else {
            if (threadIdx.x == 0) {
                // the relay may idle for up to idle_ticks, then finish the previous packet's wait
                uint32_t end = wait_word(published, (uint32_t)k, r.idle_ticks + 2 * r.timeout_ticks) ? 0u : 1u;
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
                if (!end && __hip_atomic_load(stop_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) end = 1;
                stop = end;
            }
            __syncthreads();
            if (!stop)
                for (uint32_t i = threadIdx.x; i < kWords; i += kBlockThreads)
                    pk[i] = __hip_atomic_load(mirror + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __syncthreads();
        }
        if (stop) break;

        const LaunchArgs& a = *(const LaunchArgs*)pk;
        const uint8_t* prog = a.prog;
        ProgramHeader h;
        h.ndesc = cld<uint32_t>(prog, offsetof(ProgramHeader, ndesc));
        h.ntiles = cld<uint32_t>(prog, offsetof(ProgramHeader, ntiles));
        h.nstate = cld<uint32_t>(prog, offsetof(ProgramHeader, nstate));
        h.off_desc = cld<uint64_t>(prog, offsetof(ProgramHeader, off_desc));
        h.off_operand = cld<uint64_t>(prog, offsetof(ProgramHeader, off_operand));
        h.off_dep = cld<uint64_t>(prog, offsetof(ProgramHeader, off_dep));
        h.off_tile_desc = cld<uint64_t>(prog, offsetof(ProgramHeader, off_tile_desc));
        h.off_aux = cld<uint64_t>(prog, offsetof(ProgramHeader, off_aux));
        const bool has_deps = (cld<uint32_t>(prog, offsetof(ProgramHeader, flags)) & PF_HAS_DEPS) != 0u;
        uint32_t* const state = a.state;
        const uint64_t* bufs = pk + offsetof(LaunchArgs, bufs) / 8;
        Shared sh;
        sh.state = state;
        sh.error = r.error;
        sh.timeout = r.timeout_ticks;
        for (uint32_t t = a.tile_begin + wave; t < a.tile_end; t += nworkers) {
            if (has_deps && load_relaxed(&r.error->code) != 0u) break;
            uint64_t unused = 0;
            if (!run_tile<kKindGeneric>(sh, prog, h, t, lane, bufs, false, unused)) break;
        }

        // this workgroup's stores and counter updates are complete and visible device-wide
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __syncthreads();
        if (threadIdx.x == 0) {
            const uint32_t prev = __hip_atomic_fetch_add(arrived, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
            last_block = (prev == gridDim.x - 1) ? 1u : 0u;
        }
        __syncthreads();
        if (last_block) {
            if (has_deps)
                for (uint32_t i = threadIdx.x; i < h.nstate; i += kBlockThreads)
                    __hip_atomic_store(state + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (threadIdx.x == 0) {
                const uint32_t code = load_relaxed(&r.error->code);
                if (code != 0u) {
                    // only this thread writes the record (packets complete one at a time), so plain
                    // stores suffice: no atomic read-modify-write goes to host memory
                    if (__hip_atomic_load(&r.q->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) == 0u) {
                        __hip_atomic_store(&r.q->error, code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                        __hip_atomic_store(&r.q->err_desc, load_relaxed(&r.error->desc), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_SYSTEM);
                        __hip_atomic_store(&r.q->err_tile, load_relaxed(&r.error->tile), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_SYSTEM);
                    }
                    __hip_atomic_store(&r.error->code, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                __hip_atomic_store(arrived, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                // results and counters reach memory before the host or the relay sees the number
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
                __hip_atomic_store(&r.q->done_seq, k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                __hip_atomic_store(finished, (uint32_t)k, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        if (relay) {
            // Wait until every workgroup has finished packet k (the next packet may reuse its
            // counters). Meanwhile, if packet k + 1 is already at the doorbell, bring its
            // arguments into LDS and the other mirror, so that its PCIe round trips overlap the
            // others' work on packet k. (pk is free: this workgroup has finished packet k.)
            ResidentSlot* next = &r.q->slots[k % kResidentSlots];
            uint64_t* const next_mirror = r.mirror + ((k + 1) & 1) * kWords;
            uint32_t nap = 1;
            const uint64_t t0 = wall_clock64();
            for (;;) {
                if (threadIdx.x == 0) {
                    uint32_t g = 0;  // 1 = packet k finished, 2 = gave up waiting
                    if (last_block || __hip_atomic_load(finished, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)k)
                        g = 1;
                    else if (wall_clock64() - t0 > r.timeout_ticks)
                        g = 2;
                    uint32_t f = 0;  // 1 = fetch packet k + 1 now, 2 = it is the stop request
                    if (!ahead) {
                        const uint64_t v = __hip_atomic_load(&next->seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                        if ((v & ~kResidentStop) == k + 1) {
                            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
                            f = (v & kResidentStop) ? 2u : 1u;
                        }
                    }
                    sig = g;
                    fetch = f;
                }
                __syncthreads();
                const uint32_t g = sig, f = fetch;
                if (f == 1u) {
                    const uint64_t* from = (const uint64_t*)&next->args;
                    for (uint32_t i = threadIdx.x; i < kWords; i += kBlockThreads) {
                        const uint64_t w = __hip_atomic_load(from + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                        pk[i] = w;
                        __hip_atomic_store(next_mirror + i, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                    __builtin_amdgcn_s_waitcnt(0);
                }
                __syncthreads();
                if (threadIdx.x == 0) {
                    if (f != 0u) {
                        ahead = 1;
                        ahead_stop = f == 2u ? 1u : 0u;
                    }
                    if (g == 2u) {
                        stop = 1;
                        why = RESIDENT_EXIT_WORKGROUPS;
                    }
                    if (g == 0u) backoff(nap, 4);
                }
                if (g != 0u) break;
            }
            if (threadIdx.x == 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            __syncthreads();
            if (stop) {
                // release the others from their wait for packet k + 1
                if (threadIdx.x == 0) {
                    __hip_atomic_store(stop_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(published, (uint32_t)(k + 1), __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
                }
                break;
            }
        }
    }
    if (threadIdx.x == 0 && relay) __hip_atomic_store(&r.q->exited, why, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// A program of one step needs no device image: its step travels inside the launch packet
// with every operand already resolved to an address (the analogue of the express doorbell,
// where the work request itself is the doorbell write and nothing is fetched first).
template <int KIND>
__global__ void __launch_bounds__(kBlockThreads) hccl_executor_inline(InlineArgs a) {
    const uint32_t lane = __lane_id();
    const uint32_t wave = uni(blockIdx.x * kWavesPerBlock + (threadIdx.x / kWaveSize));
    const char* kargs = (const char*)__builtin_amdgcn_kernarg_segment_ptr();
    const uint64_t* srcs = (const uint64_t*)(kargs + offsetof(InlineArgs, src));
    const uint64_t* dsts = (const uint64_t*)(kargs + offsetof(InlineArgs, dst));
    TileOps ops;
    ops.nsrc = a.nsrc;
    ops.ndst = a.ndst;
    ops.group = a.group;
    ops.fold = a.fold;
    ops.requant = a.requant;
    const uint64_t te = a.tile_elems;
    for (uint32_t t = wave; t < a.ntiles; t += a.nworkers) {
        const uint64_t e0 = (uint64_t)t * te;
        const uint32_t n = (uint32_t)((a.nelem - e0 < te) ? (a.nelem - e0) : te);
        ops.src = lane < ops.nsrc ? srcs[lane] + e0 * (lane == 0 ? a.es_first : a.es_rest) : 0;
        ops.dst = lane < ops.ndst ? dsts[lane] + e0 * a.es_out : 0;
        const bool misaligned = (lane < ops.nsrc && (ops.src & 15u)) || (lane < ops.ndst && (ops.dst & 15u));
        exec_tile<KIND>(a.op, a.sig, a.redop, a.es_first, ops, n, __ballot(misaligned) == 0ull, lane);
    }
}

__global__ void hccl_fill_u32(uint32_t* p, uint64_t n, uint32_t v) {
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i < n; i += (uint64_t)gridDim.x * blockDim.x) p[i] = v;
}

}  // namespace

hipError_t launch_executor_inline(const InlineArgs& a, uint32_t blocks, int kind, hipStream_t stream) {
    switch (kind) {
        case SIG_BF16: hipLaunchKernelGGL(hccl_executor_inline<SIG_BF16>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case SIG_FP16: hipLaunchKernelGGL(hccl_executor_inline<SIG_FP16>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case SIG_FP32: hipLaunchKernelGGL(hccl_executor_inline<SIG_FP32>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case SIG_INT32: hipLaunchKernelGGL(hccl_executor_inline<SIG_INT32>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case kKindCopyOnly:
            hipLaunchKernelGGL(hccl_executor_inline<kKindCopyOnly>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
        case kKindCopyAligned:
            hipLaunchKernelGGL(hccl_executor_inline<kKindCopyAligned>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
        default:
            hipLaunchKernelGGL(hccl_executor_inline<kKindGeneric>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
    }
    return hipGetLastError();
}

int executor_block_threads() { return kBlockThreads; }

size_t workspace_bytes() { return kWorkspaceBytes; }

// Device address of the static workspace on the current device, looked up once per device
// and kept for the rest of the process.
hipError_t workspace_address(void** ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}
int executor_waves_per_block() { return kWavesPerBlock; }

// kind: a plain signature (SIG_BF16 .. SIG_INT32) for SUM-only programs of that signature,
// kKindCopyOnly, or anything else for the generic kernel.
hipError_t launch_executor(const LaunchArgs& a, uint32_t blocks, int kind, hipStream_t stream) {
    switch (kind) {
        case SIG_BF16: hipLaunchKernelGGL(hccl_executor<SIG_BF16>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case SIG_FP16: hipLaunchKernelGGL(hccl_executor<SIG_FP16>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case SIG_FP32: hipLaunchKernelGGL(hccl_executor<SIG_FP32>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case SIG_INT32: hipLaunchKernelGGL(hccl_executor<SIG_INT32>, dim3(blocks), dim3(kBlockThreads), 0, stream, a); break;
        case kKindCopyOnly:
            hipLaunchKernelGGL(hccl_executor<kKindCopyOnly>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
        case kKindCopyAligned:
            hipLaunchKernelGGL(hccl_executor<kKindCopyAligned>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
        case kKindDynamic:
            hipLaunchKernelGGL(hccl_executor<kKindDynamic>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
        default:
            hipLaunchKernelGGL(hccl_executor<kKindGeneric>, dim3(blocks), dim3(kBlockThreads), 0, stream, a);
            break;
    }
    return hipGetLastError();
}

hipError_t launch_signal(uint64_t* word, uint64_t value, const ErrorRecord* err, hipStream_t stream) {
    hipLaunchKernelGGL(hccl_signal, dim3(1), dim3(64), 0, stream, word, value, err);
    return hipGetLastError();
}

hipError_t launch_resident(const ResidentArgs& r, uint32_t blocks, hipStream_t stream) {
    hipLaunchKernelGGL(hccl_resident, dim3(blocks), dim3(kBlockThreads), 0, stream, r);
    return hipGetLastError();
}

hipError_t resident_occupancy(int* blocks_per_cu) {
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_resident, kBlockThreads, 0);
}

hipError_t launch_fill_u32(uint32_t* p, uint64_t n, uint32_t v, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    uint64_t blocks = (n + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(hccl_fill_u32, dim3((uint32_t)blocks), dim3(256), 0, stream, p, n, v);
    return hipGetLastError();
}

// Resident blocks per CU of the kernel of one kind.
hipError_t executor_occupancy(int kind, int* blocks_per_cu) {
    switch (kind) {
        case SIG_BF16: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<SIG_BF16>, kBlockThreads, 0);
        case SIG_FP16: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<SIG_FP16>, kBlockThreads, 0);
        case SIG_FP32: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<SIG_FP32>, kBlockThreads, 0);
        case SIG_INT32: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<SIG_INT32>, kBlockThreads, 0);
        case kKindCopyOnly: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<kKindCopyOnly>, kBlockThreads, 0);
        case kKindCopyAligned: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<kKindCopyAligned>, kBlockThreads, 0);
        case kKindDynamic: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<kKindDynamic>, kBlockThreads, 0);
        default: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, hccl_executor<kKindGeneric>, kBlockThreads, 0);
    }
}

}  // namespace hccl
