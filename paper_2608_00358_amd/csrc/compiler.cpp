// compiler.cpp -- lowering, fusion and packing of descriptor programs (host only).
//
// Lowerings write out the schedules the paper describes (Section III-B-2: the ring AllReduce
// built from per-hop receive/compute/send steps with dependencies; Section V-D: topology-
// aware two-level schedules that keep most traffic inside a group of consecutive ranks).
// On one GPU a "send" from rank a to rank b is a read of a's buffer by the step that writes
// b's buffer, so a hop becomes a COPY or REDUCE descriptor with a dependency id on the step
// that produced its input.
//
// Every reduction visits contributors in ascending rank order (two-level: ascending inside
// each group, then ascending over groups), so results never depend on the schedule.
#include "compiler.h"

#include <algorithm>
#include <cstring>
#include <unordered_map>

namespace hccl {

namespace {

constexpr uint64_t kDefaultChunkBytes = 1ull << 20;
// Tile defaults measured on MI355X: copies move 8 KiB per ticket; reductions read 32 KiB
// per ticket but never less than 1024 elements (wide two-level steps).
constexpr uint32_t kDefaultCopyTileBytes = 8u * 1024u;
constexpr uint32_t kDefaultReduceTileBytes = 32u * 1024u;
constexpr uint64_t kMinReduceTileElems = 1024;
// Programs with dependencies pay a release fence per signalling tile: larger tiles. A small
// dependent program (a few chains of long steps) would then leave most wavefronts idle, so its
// tiles are halved, down to 32 KiB read, until it has at least kDependentMinTiles (measured on
// the ring all-reduce P=4 x 2^20 fp32, 64 KiB chunks, unfused: 384 tiles 117 us, 1536 tiles
// 93 us; 3072 tiles 133 us and smaller ones slower still, as fences multiply).
constexpr uint32_t kDefaultDependentTileBytes = 128u * 1024u;
constexpr uint32_t kMinDependentTileBytes = 32u * 1024u;
constexpr uint64_t kDependentMinTiles = 1024;
// A copy to this many destinations or more reads up to 32 KiB per tile, as long as its phase
// keeps about 256 tiles: each tile writes its bytes to every destination, so a few long tiles
// beat many short ones. Measured with one wavefront per tile on the copy phase of the two-level
// all-reduce of 64 ranks (every 1/64 sub-shard to 63 ranks): tiles of the phase's bytes / 1024
// -> / 256 took 8 MiB per rank 222 -> 183 us, 4 MiB 109 -> 102 us; at 32 MiB per rank 32 KiB
// tiles (1 024) 736-754 us against 64 KiB 745-762 us and 128 KiB 819-836 us; the all-gather of
// P = 64 x 512 KiB bf16 blocks 396-400 us with 32 KiB tiles, 418-424 with 64 KiB, 543-550 with
// 128 KiB, 515-525 with 8 KiB.
constexpr size_t kWideCopyDsts = 8;
constexpr uint64_t kWideCopyTileBytes = 32u * 1024u;
constexpr uint64_t kWideCopyTargetTiles = 256;
// Small collectives are latency bound: cut them into at least this many tiles (down to
// one vector per lane) so that many wavefronts share the work.
constexpr uint64_t kSmallTargetTiles = 2048;
constexpr uint32_t kWaveStepElems = kWaveSize * kVecElems;  // 512: one vector per lane
constexpr uint64_t kShardAlignElems = 64;                      // 128 B of bf16, 256 B of fp32
// Static tiles (slots) of the copy step of an AllToAllvDynamic: slot k moves dynamic tiles k,
// k + slots, ... Every slot plans the exchange itself, so more slots cost more for an exchange
// far below its capacities, while fewer leave each slot a longer run of tiles. The launch has
// one wavefront per slot; rows + ids of the 8-rank 2^18-row exchange, full / all counts zero:
// 4 096 + 1 088 slots 197-198 / 8 us, 16 384 + 1 088 194 / 14 us, 32 768 + 1 088 192-193 /
// 23-24 us, 65 536 + 1 088 190 / 44 us.
constexpr uint32_t kDynamicSlots = 32768;

// Type of partials that leave registers: FP32 for floating sums (one rounding at the end),
// the buffer type when every partial is re-quantised, or for MAX / MIN (exact in any type).
uint32_t acc_dtype(const CollectiveSpec& s) {
    if (s.dtype == DT_INT32) return DT_INT32;
    if (s.redop != RO_SUM || s.requant) return (uint32_t)s.dtype;
    return DT_FP32;
}

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

// Contributors of an element of shard (or block) c in fold order.
std::vector<int> contributor_order(const CollectiveSpec& s, int c) {
    const int P = s.P;
    std::vector<int> v(P);
    for (int k = 0; k < P; ++k) {
        if (s.order == ORDER_RING) {
            v[k] = (c + 1 + k) % P;
        } else if (s.order == ORDER_HALVING) {
            int r = 0;  // bit reversal of k: adjacent list entries differ in bit P/2, pairs of
            for (int b = 1, t = P >> 1; b < P; b <<= 1, t >>= 1)  // pairs in bit P/4, ...
                if (k & b) r |= t;
            v[k] = r;
        } else {
            v[k] = k;
        }
    }
    return v;
}

uint64_t chunk_elems(const CollectiveSpec& s) {
    uint64_t bytes = s.chunk_bytes ? s.chunk_bytes : kDefaultChunkBytes;
    uint64_t c = bytes / dtype_size(s.dtype);
    c = (c / kShardAlignElems) * kShardAlignElems;
    return std::max<uint64_t>(c, kShardAlignElems);
}

Operand opnd(uint32_t buf, uint32_t dtype, uint64_t elem_offset) {
    Operand o;
    o.buf = buf;
    o.dtype = dtype;
    o.offset = elem_offset * dtype_size(dtype);
    return o;
}

struct Builder {
    HostProgram& prog;
    uint32_t add(uint8_t op, uint8_t redop, uint64_t nelem, std::vector<Operand> srcs,
                 std::vector<Operand> dsts, std::vector<Dep> deps = {}, uint16_t group = 0) {
        HostDesc d;
        d.op = op;
        d.redop = redop;
        d.nelem = nelem;
        d.group = group;
        d.srcs = std::move(srcs);
        d.dsts = std::move(dsts);
        d.deps = std::move(deps);
        prog.descs.push_back(std::move(d));
        return (uint32_t)(prog.descs.size() - 1);
    }
};

Dep tile_dep(uint32_t d) { return Dep{d, DEP_TILE, 0, 0}; }

template <typename F>
void for_chunks(uint64_t begin, uint64_t end, uint64_t C, F&& f) {
    uint32_t j = 0;
    for (uint64_t o = begin; o < end; o += C, ++j) f(j, o, std::min(C, end - o));
}

// ---------------------------------------------------------------------------- DIRECT
// One step per chunk: read every contributor, write every destination (the one-shot,
// all-to-all style schedule of the PE collective kernels for small messages, Section V-F-3).
void lower_direct(const CollectiveSpec& s, HostProgram& p) {
    Builder b{p};
    const int P = s.P;
    const uint64_t C = chunk_elems(s);
    const uint32_t dt = (uint32_t)s.dtype;
    const uint32_t fold = (s.order == ORDER_HALVING) ? FOLD_PAIRWISE : FOLD_LIST;
    auto reduce_step = [&](uint64_t n, const std::vector<int>& order, uint64_t src_elem, std::vector<Operand> dst) {
        std::vector<Operand> src;
        for (int r : order) src.push_back(opnd(send_buf(r), dt, src_elem));
        uint32_t i = b.add(OP_REDUCE, (uint8_t)s.redop, n, src, std::move(dst));
        p.descs[i].fold = fold;
    };
    if (s.coll == COLL_ALLREDUCE) {
        // the ring order rotates per shard, so chunks never straddle a shard boundary then
        const uint64_t q = (s.order == ORDER_RING) ? shard_size(s.count, P) : s.count;
        for (uint64_t lo = 0, c = 0; lo < s.count; lo += q, ++c) {
            const std::vector<int> order = contributor_order(s, (int)c);
            for_chunks(lo, std::min(s.count, lo + q), C, [&](uint32_t, uint64_t o, uint64_t n) {
                std::vector<Operand> dst;
                for (int r = 0; r < P; ++r) dst.push_back(opnd(recv_buf(P, r), dt, o));
                reduce_step(n, order, o, dst);
            });
        }
    } else if (s.coll == COLL_REDUCE_SCATTER) {
        const uint64_t M = s.count;
        for (int c = 0; c < P; ++c) {
            const std::vector<int> order = contributor_order(s, c);
            for_chunks(0, M, C, [&](uint32_t, uint64_t o, uint64_t n) {
                reduce_step(n, order, (uint64_t)c * M + o, {opnd(recv_buf(P, c), dt, o)});
            });
        }
    } else if (s.coll == COLL_ALLGATHER) {
        const uint64_t M = s.count;
        for (int q = 0; q < P; ++q) {
            for_chunks(0, M, C, [&](uint32_t, uint64_t o, uint64_t n) {
                std::vector<Operand> dst;
                for (int r = 0; r < P; ++r) dst.push_back(opnd(recv_buf(P, r), dt, (uint64_t)q * M + o));
                b.add(OP_COPY, RO_SUM, n, {opnd(send_buf(q), dt, o)}, dst);
            });
        }
    }
    p.algo = ALGO_DIRECT;
}

// ------------------------------------------------------------------------------ RING
// Reduce chain of one chunk: step t (t = 1 .. P-1) folds contributor t into the partial of
// contributors 0 .. t-1. Partials live in scratch in the accumulation type; the last step
// rounds into `final_dst`. Steps of all chunks are emitted step-major so every chunk's step
// t is available while step t+1 waits only for the same tile of its own chain.
struct Chain {
    int owner = 0;        // shard / block the chain reduces (fixes the ring order's start)
    uint64_t src_elem;    // element offset of the chunk in every send buffer
    uint64_t nelem;
    Operand final_dst;
    uint64_t scratch_elem;  // element offset of the partial in scratch (accumulation type)
    uint32_t last = 0;      // descriptor of the final step
    uint32_t prev = 0;
};

void emit_reduce_chains(const CollectiveSpec& s, HostProgram& p, std::vector<Chain>& chains) {
    Builder b{p};
    const int P = s.P;
    const uint32_t dt = (uint32_t)s.dtype;
    const uint32_t acc = acc_dtype(s);
    if (P == 1) {
        for (auto& ch : chains)
            ch.last = b.add(OP_REDUCE, (uint8_t)s.redop, ch.nelem, {opnd(send_buf(0), dt, ch.src_elem)},
                            {ch.final_dst});
        return;
    }
    std::vector<std::vector<int>> order(P);
    for (int c = 0; c < P; ++c) order[c] = contributor_order(s, c);
    for (int t = 1; t < P; ++t) {
        for (auto& ch : chains) {
            const std::vector<int>& seq = order[ch.owner];
            Operand partial = opnd(scratch_buf(P), acc, ch.scratch_elem);
            std::vector<Operand> src;
            if (t == 1) src.push_back(opnd(send_buf(seq[0]), dt, ch.src_elem));
            else src.push_back(partial);
            src.push_back(opnd(send_buf(seq[t]), dt, ch.src_elem));
            Operand dst = (t == P - 1) ? ch.final_dst : partial;
            std::vector<Dep> deps;
            if (t > 1) deps.push_back(tile_dep(ch.prev));
            ch.prev = b.add(OP_REDUCE, (uint8_t)s.redop, ch.nelem, src, {dst}, deps);
            if (t == P - 1) ch.last = ch.prev;
        }
    }
}

void lower_ring(const CollectiveSpec& s, HostProgram& p) {
    Builder b{p};
    const int P = s.P;
    const uint64_t C = chunk_elems(s);
    const uint32_t dt = (uint32_t)s.dtype;
    const uint32_t acc = acc_dtype(s);

    if (s.coll == COLL_ALLGATHER) {
        // hop 0 places block q in rank q's output; hop h forwards it from rank q+h-1 to q+h.
        const uint64_t M = s.count;
        struct Hop { int q; uint64_t o, n; uint32_t prev; };
        std::vector<Hop> hops;
        for (int q = 0; q < P; ++q)
            for_chunks(0, M, C, [&](uint32_t, uint64_t o, uint64_t n) { hops.push_back({q, o, n, 0}); });
        for (auto& h : hops)
            h.prev = b.add(OP_COPY, RO_SUM, h.n, {opnd(send_buf(h.q), dt, h.o)},
                           {opnd(recv_buf(P, h.q), dt, (uint64_t)h.q * M + h.o)});
        for (int step = 1; step < P; ++step) {
            for (auto& h : hops) {
                int from = (h.q + step - 1) % P, to = (h.q + step) % P;
                uint64_t at = (uint64_t)h.q * M + h.o;
                h.prev = b.add(OP_COPY, RO_SUM, h.n, {opnd(recv_buf(P, from), dt, at)},
                               {opnd(recv_buf(P, to), dt, at)}, {tile_dep(h.prev)});
            }
        }
        p.algo = ALGO_RING;
        return;
    }

    std::vector<Chain> chains;
    std::vector<int> owner;
    if (s.coll == COLL_REDUCE_SCATTER) {
        const uint64_t M = s.count;
        for (int c = 0; c < P; ++c)
            for_chunks(0, M, C, [&](uint32_t, uint64_t o, uint64_t n) {
                Chain ch;
                ch.owner = c;
                ch.src_elem = (uint64_t)c * M + o;
                ch.nelem = n;
                ch.final_dst = opnd(recv_buf(P, c), dt, o);
                ch.scratch_elem = (uint64_t)c * M + o;
                chains.push_back(ch);
                owner.push_back(c);
            });
        p.scratch_bytes = (P > 2) ? (uint64_t)P * M * dtype_size(acc) : 0;
    } else {  // allreduce: owner c reduces shard c, then the result travels around the ring
        const uint64_t q = shard_size(s.count, P);
        for (int c = 0; c < P; ++c) {
            uint64_t lo = std::min(s.count, (uint64_t)c * q), hi = std::min(s.count, lo + q);
            for_chunks(lo, hi, C, [&](uint32_t, uint64_t o, uint64_t n) {
                Chain ch;
                ch.owner = c;
                ch.src_elem = o;
                ch.nelem = n;
                ch.final_dst = opnd(recv_buf(P, c), dt, o);
                ch.scratch_elem = o;
                chains.push_back(ch);
                owner.push_back(c);
            });
        }
        p.scratch_bytes = (P > 2) ? s.count * dtype_size(acc) : 0;
    }
    emit_reduce_chains(s, p, chains);

    if (s.coll == COLL_ALLREDUCE) {
        for (int step = 1; step < P; ++step) {
            for (size_t i = 0; i < chains.size(); ++i) {
                Chain& ch = chains[i];
                int from = (owner[i] + step - 1) % P, to = (owner[i] + step) % P;
                ch.last = b.add(OP_COPY, RO_SUM, ch.nelem, {opnd(recv_buf(P, from), dt, ch.src_elem)},
                                {opnd(recv_buf(P, to), dt, ch.src_elem)}, {tile_dep(ch.last)});
            }
        }
    }
    p.algo = ALGO_RING;
}

// ------------------------------------------------------------------------------- RHD
// Recursive halving reduce-scatter (and recursive doubling all-gather) for P = 2^L ranks.
// The vector is cut into P blocks; block b ends at rank b. At halving step j (distance
// d = P >> (j+1)) rank r keeps the blocks that agree with r on every bit handled so far; for
// each kept block it combines its own value with the value of partner r ^ d, which kept the
// same block one step earlier. Partials live in scratch slot (r, b) in the accumulation type;
// the last step writes the owner's receive buffer. The tree this builds for every element
// pairs ranks differing in bit P/2 first, then bit P/4, ..., then bit 1. Doubling step j
// (distance d = 1 << j) copies the d blocks a rank holds to its partner r ^ d.
void lower_rhd(const CollectiveSpec& s, HostProgram& p) {
    Builder b{p};
    const int P = s.P;
    const uint64_t C = chunk_elems(s);
    const uint32_t dt = (uint32_t)s.dtype;
    const uint32_t acc = acc_dtype(s);
    const bool ag_only = s.coll == COLL_ALLGATHER;
    // block geometry: element offset of block b in a send buffer / in a receive buffer
    const uint64_t N = s.count;
    const uint64_t q = (s.coll == COLL_ALLREDUCE) ? shard_size(N, P) : N;
    auto blo = [&](int blk) { return std::min<uint64_t>((uint64_t)blk * q, s.coll == COLL_ALLREDUCE ? N : (uint64_t)P * N); };
    auto bhi = [&](int blk) { return std::min<uint64_t>(blo(blk) + q, s.coll == COLL_ALLREDUCE ? N : (uint64_t)P * N); };
    // receive-side element offset of block b: all-reduce and all-gather keep the send layout;
    // reduce-scatter writes its block at offset 0 of the owner's buffer
    auto rlo = [&](int blk) { return s.coll == COLL_REDUCE_SCATTER ? 0 : blo(blk); };

    // producer of the value rank r holds for (block, chunk offset), per step
    std::vector<std::unordered_map<uint64_t, uint32_t>> prev(P), next(P);
    auto key = [&](int blk, uint64_t o) { return ((uint64_t)blk << 40) | (o - blo(blk)); };

    if (!ag_only) {
        int steps = 0;
        while ((1 << steps) < P) ++steps;
        uint64_t mask = 0;
        for (int j = 0; j < steps; ++j) {
            const int d = P >> (j + 1);
            mask |= (uint64_t)d;
            for (int r = 0; r < P; ++r) next[r].clear();
            for (int r = 0; r < P; ++r) {
                const int partner = r ^ d;
                for (int blk = 0; blk < P; ++blk) {
                    if (((uint64_t)blk & mask) != ((uint64_t)r & mask)) continue;
                    const bool last = (j == steps - 1);
                    for_chunks(blo(blk), bhi(blk), C, [&](uint32_t, uint64_t o, uint64_t n) {
                        const uint64_t so = (uint64_t)(r * P + blk) * q + (o - blo(blk));
                        const uint64_t po = (uint64_t)(partner * P + blk) * q + (o - blo(blk));
                        std::vector<Operand> src;
                        std::vector<Dep> deps;
                        if (j == 0) {
                            src.push_back(opnd(send_buf(r), dt, o));
                            src.push_back(opnd(send_buf(partner), dt, o));
                        } else {
                            src.push_back(opnd(scratch_buf(P), acc, so));
                            src.push_back(opnd(scratch_buf(P), acc, po));
                            deps.push_back(tile_dep(prev[r].at(key(blk, o))));
                            deps.push_back(tile_dep(prev[partner].at(key(blk, o))));
                        }
                        Operand dst = last ? opnd(recv_buf(P, r), dt, rlo(blk) + (o - blo(blk)))
                                           : opnd(scratch_buf(P), acc, so);
                        next[r][key(blk, o)] = b.add(OP_REDUCE, (uint8_t)s.redop, n, src, {dst}, deps);
                    });
                }
            }
            prev.swap(next);
        }
        p.scratch_bytes = (steps > 1) ? (uint64_t)P * P * q * dtype_size(acc) : 0;
        if (P == 1) {
            for_chunks(blo(0), bhi(0), C, [&](uint32_t, uint64_t o, uint64_t n) {
                prev[0][key(0, o)] = b.add(OP_REDUCE, (uint8_t)s.redop, n, {opnd(send_buf(0), dt, o)},
                                           {opnd(recv_buf(P, 0), dt, rlo(0) + (o - blo(0)))});
            });
        }
    } else {
        // all-gather: every rank first places its own block
        for (int r = 0; r < P; ++r)
            for_chunks(0, N, C, [&](uint32_t, uint64_t o, uint64_t n) {
                prev[r][key(r, (uint64_t)r * N + o)] =
                    b.add(OP_COPY, RO_SUM, n, {opnd(send_buf(r), dt, o)}, {opnd(recv_buf(P, r), dt, (uint64_t)r * N + o)});
            });
    }

    if (s.coll != COLL_REDUCE_SCATTER) {
        // doubling: at distance d, rank r holds the d blocks of its aligned group and sends them
        for (int d = 1; d < P; d <<= 1) {
            for (int r = 0; r < P; ++r) next[r] = prev[r];
            for (int r = 0; r < P; ++r) {
                const int partner = r ^ d;
                const int base = r & ~(d - 1);
                for (int blk = base; blk < base + d; ++blk) {
                    for_chunks(blo(blk), bhi(blk), C, [&](uint32_t, uint64_t o, uint64_t n) {
                        const uint32_t src_desc = prev[r].at(key(blk, o));
                        next[partner][key(blk, o)] =
                            b.add(OP_COPY, RO_SUM, n, {opnd(recv_buf(P, r), dt, o)}, {opnd(recv_buf(P, partner), dt, o)},
                                  {tile_dep(src_desc)});
                    });
                }
            }
            prev.swap(next);
        }
    }
    p.algo = ALGO_RHD;
}

// ------------------------------------------------------------------------- TWO_LEVEL
// P = G groups x L consecutive ranks. Shard k of the vector belongs to local rank k of every
// group and is cut into G sub-shards; sub-shard (k, g) is owned by local rank k of group g.
// Phase 1 (inside each group, reduce-scatter): the L contributors of every element are folded
// into an FP32 partial per group. Phase 2 (across groups, the all-reduce of shard k among the
// local-k ranks as reduce-scatter + all-gather): the G partials of sub-shard (k, g) are folded
// in ascending group order, rounded, and written to its owner; the owner forwards it to local
// rank k of the other groups. Phase 3 (inside each group, all-gather): local rank k forwards
// shard k to the other L-1 ranks of its group.
void lower_two_level(const CollectiveSpec& s, HostProgram& p) {
    Builder b{p};
    const int P = s.P, L = s.group_size, G = P / L;
    const uint64_t N = s.count, C = chunk_elems(s);
    const uint32_t dt = (uint32_t)s.dtype;
    const uint32_t acc = acc_dtype(s);
    const uint64_t q = shard_size(N, L);
    struct Piece { int k, g; uint64_t o, n; };
    std::vector<Piece> pieces;
    for (int k = 0; k < L; ++k) {
        const uint64_t lo = std::min(N, (uint64_t)k * q), hi = std::min(N, lo + q);
        const uint64_t qs = shard_size(hi - lo, G);
        for (int g = 0; g < G; ++g) {
            const uint64_t slo = std::min(hi, lo + (uint64_t)g * qs), shi = std::min(hi, slo + qs);
            for_chunks(slo, shi, C, [&](uint32_t, uint64_t o, uint64_t n) { pieces.push_back({k, g, o, n}); });
        }
    }
    auto rank = [&](int g, int m) { return g * L + m; };
    std::vector<std::vector<uint32_t>> rs(pieces.size(), std::vector<uint32_t>(G));
    for (int h = 0; h < G; ++h) {
        for (size_t i = 0; i < pieces.size(); ++i) {
            const Piece& pc = pieces[i];
            std::vector<Operand> src;
            for (int m = 0; m < L; ++m) src.push_back(opnd(send_buf(rank(h, m)), dt, pc.o));
            rs[i][h] = b.add(OP_REDUCE, (uint8_t)s.redop, pc.n, src,
                             {opnd(scratch_buf(P), acc, (uint64_t)h * N + pc.o)});
        }
    }
    std::vector<uint32_t> inter(pieces.size()), fwd(pieces.size());
    for (size_t i = 0; i < pieces.size(); ++i) {
        const Piece& pc = pieces[i];
        std::vector<Operand> src;
        std::vector<Dep> deps;
        for (int h = 0; h < G; ++h) {
            src.push_back(opnd(scratch_buf(P), acc, (uint64_t)h * N + pc.o));
            deps.push_back(tile_dep(rs[i][h]));
        }
        inter[i] = b.add(OP_REDUCE, (uint8_t)s.redop, pc.n, src, {opnd(recv_buf(P, rank(pc.g, pc.k)), dt, pc.o)}, deps);
    }
    for (size_t i = 0; i < pieces.size(); ++i) {
        const Piece& pc = pieces[i];
        fwd[i] = inter[i];
        if (G == 1) continue;
        std::vector<Operand> dst;
        for (int h = 0; h < G; ++h)
            if (h != pc.g) dst.push_back(opnd(recv_buf(P, rank(h, pc.k)), dt, pc.o));
        fwd[i] = b.add(OP_COPY, RO_SUM, pc.n, {opnd(recv_buf(P, rank(pc.g, pc.k)), dt, pc.o)}, dst,
                       {tile_dep(inter[i])});
    }
    if (L > 1) {
        for (int h = 0; h < G; ++h) {
            for (size_t i = 0; i < pieces.size(); ++i) {
                const Piece& pc = pieces[i];
                std::vector<Operand> dst;
                for (int m = 0; m < L; ++m)
                    if (m != pc.k) dst.push_back(opnd(recv_buf(P, rank(h, m)), dt, pc.o));
                b.add(OP_COPY, RO_SUM, pc.n, {opnd(recv_buf(P, rank(h, pc.k)), dt, pc.o)}, dst,
                      {tile_dep(h == pc.g ? inter[i] : fwd[i])});
            }
        }
    }
    p.scratch_bytes = (uint64_t)G * N * dtype_size(acc);
    p.algo = ALGO_TWO_LEVEL;
}

// ------------------------------------------------------------------------- ALLTOALLV
// Every non-empty (source, destination) block becomes COPY steps of at most one chunk; the
// steps are ordered largest first so the long blocks start early (Section IV-A: AllToAllv
// spread across parallel engines), and equal ones destination by destination: launches start
// their tiles in program order, so at any moment the chip fills one receive buffer in order
// while it reads from every send buffer (grouped AllToAllv of 8 ranks x 2^18 embedding rows,
// source-major 182.8-184.2 us, destination-major 181.0-182.5 us).
void lower_alltoallv(const CollectiveSpec& s, HostProgram& p) {
    Builder b{p};
    const int P = s.P;
    const uint32_t dt = (uint32_t)s.dtype;
    const uint64_t C = chunk_elems(s);
    struct Piece { int src, dst; uint64_t so, ro, n; };
    std::vector<Piece> pieces;
    for (int dst = 0; dst < P; ++dst) {
        for (int src = 0; src < P; ++src) {
            uint64_t n = s.sendcounts[(size_t)src * P + dst];
            uint64_t so = s.sdispls[(size_t)src * P + dst];
            uint64_t ro = s.rdispls[(size_t)dst * P + src];
            for (uint64_t o = 0; o < n; o += C) pieces.push_back({src, dst, so + o, ro + o, std::min(C, n - o)});
        }
    }
    std::stable_sort(pieces.begin(), pieces.end(), [](const Piece& a, const Piece& c) { return a.n > c.n; });
    for (const Piece& pc : pieces)
        b.add(OP_COPY, RO_SUM, pc.n, {opnd(send_buf(pc.src), dt, pc.so)}, {opnd(recv_buf(P, pc.dst), dt, pc.ro)});
    p.algo = ALGO_DIRECT;
}

// ------------------------------------------------------------------ ALLTOALLV DYNAMIC
// Device-resident AllToAllv (Section IV-B-2): the host compiles the program once for the
// capacities, and the layout is worked out on the device when it runs. The program is one
// step of `slots` tiles; each slot reads the count matrix (and the explicit offsets, if given)
// from device memory, checks the whole layout, and moves its share of the rows. Nothing on the
// host depends on the counts, and no slot waits for another.
void lower_alltoallv_dynamic(const CollectiveSpec& s, HostProgram& p) {
    const int P = s.P;
    DynA2A a;
    std::memset(&a, 0, sizeof a);
    a.P = (uint32_t)P;
    a.elem_bytes = dtype_size(s.dtype);
    a.send0 = send_buf(0);
    a.recv0 = recv_buf(P, 0);
    a.counts = meta_buf(P, META_COUNTS);
    a.sdispls = s.dyn_sdispls ? meta_buf(P, META_SDISPLS) : kNoBuffer;
    a.rdispls = s.dyn_rdispls ? meta_buf(P, META_RDISPLS) : kNoBuffer;
    a.recvcounts = s.dyn_recvcounts ? meta_buf(P, META_RECVCOUNTS) : kNoBuffer;
    a.row_elems = s.row_elems;
    a.send_cap = s.send_cap;
    a.recv_cap = s.recv_cap;
    a.tile_elems = dynamic_tile_elems(s);
    a.slots = dynamic_slots(s);
    p.aux.push_back(a);
    p.nmeta = kMetaPerDynamicCall;
    HostDesc copy;
    copy.op = OP_DYN_COPY;
    copy.aux = 0;
    p.descs.push_back(copy);
    p.algo = ALGO_DIRECT;
}

void dedupe_deps(HostDesc& d, uint32_t self) {
    std::vector<Dep> out;
    for (const Dep& e : d.deps) {
        if (e.desc == self) continue;
        bool merged = false;
        for (Dep& o : out) {
            if (o.desc == e.desc) {
                if (e.kind == DEP_ALL) o.kind = DEP_ALL;  // the stronger wait wins
                merged = true;
                break;
            }
        }
        if (!merged) out.push_back(e);
    }
    d.deps = std::move(out);
}

struct OperandKey {
    uint32_t buf;
    uint64_t offset;
    bool operator==(const OperandKey& o) const { return buf == o.buf && offset == o.offset; }
};
struct OperandKeyHash {
    size_t operator()(const OperandKey& k) const { return std::hash<uint64_t>()(k.offset * 131 + k.buf); }
};

}  // namespace

uint64_t shard_size(uint64_t n, int parts) {
    uint64_t q = (n + parts - 1) / parts;
    return ((q + kShardAlignElems - 1) / kShardAlignElems) * kShardAlignElems;
}

bool CollectiveSpec::operator==(const CollectiveSpec& o) const {
    return coll == o.coll && P == o.P && dtype == o.dtype && redop == o.redop && count == o.count &&
           sendcounts == o.sendcounts && sdispls == o.sdispls && recvcounts == o.recvcounts &&
           rdispls == o.rdispls && in_place == o.in_place && algo == o.algo && group_size == o.group_size &&
           chunk_bytes == o.chunk_bytes && fuse == o.fuse && tile_bytes == o.tile_bytes && order == o.order &&
           requant == o.requant && phases == o.phases && row_elems == o.row_elems && send_cap == o.send_cap && recv_cap == o.recv_cap &&
           dyn_sdispls == o.dyn_sdispls && dyn_rdispls == o.dyn_rdispls && dyn_recvcounts == o.dyn_recvcounts;
}

uint64_t dynamic_tile_elems(const CollectiveSpec& s) {
    const uint64_t tb = s.tile_bytes ? s.tile_bytes : kDefaultCopyTileBytes;
    const uint64_t te = (tb / dtype_size(s.dtype)) / kWaveStepElems * kWaveStepElems;
    return std::min<uint64_t>(std::max<uint64_t>(te, kWaveStepElems), 1ull << 30);
}

uint64_t dynamic_tile_bound(const CollectiveSpec& s) {
    // a source's pairs cover at most send_cap rows, and each pair adds at most one partial tile
    const uint64_t te = dynamic_tile_elems(s);
    const uint64_t per_source = (s.send_cap * s.row_elems + te - 1) / te + (uint64_t)s.P;
    return (uint64_t)s.P * per_source;
}

uint32_t dynamic_slots(const CollectiveSpec& s) {
    return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(kDynamicSlots, dynamic_tile_bound(s)));
}

int resolve_algo(const CollectiveSpec& s) {
    if (s.coll == COLL_ALLTOALLV || s.coll == COLL_ALLTOALLV_DYNAMIC) return ALGO_DIRECT;
    if (s.algo != ALGO_AUTO) return s.algo;
    if (s.order == ORDER_HALVING) return ALGO_RHD;
    if (s.coll == COLL_ALLREDUCE && s.order == ORDER_ASCENDING && s.group_size > 1 && s.group_size < s.P &&
        s.P % s.group_size == 0)
        return ALGO_TWO_LEVEL;
    return ALGO_RING;
}

BufferSizes buffer_sizes(const CollectiveSpec& s, uint64_t scratch_bytes) {
    BufferSizes b;
    const int P = s.P;
    const uint64_t es = dtype_size(s.dtype);
    b.bytes.assign((size_t)2 * P + 1, 0);
    for (int r = 0; r < P; ++r) {
        uint64_t sb = 0, rb = 0;
        switch (s.coll) {
            case COLL_ALLREDUCE: sb = rb = s.count * es; break;
            case COLL_REDUCE_SCATTER: sb = (uint64_t)P * s.count * es; rb = s.count * es; break;
            case COLL_ALLGATHER: sb = s.count * es; rb = (uint64_t)P * s.count * es; break;
            case COLL_ALLTOALLV_DYNAMIC: sb = s.send_cap * s.row_elems * es; rb = s.recv_cap * s.row_elems * es; break;
            default:
                for (int q = 0; q < P; ++q) {
                    sb = std::max(sb, (s.sdispls[(size_t)r * P + q] + s.sendcounts[(size_t)r * P + q]) * es);
                    rb = std::max(rb, (s.rdispls[(size_t)r * P + q] + s.recvcounts[(size_t)r * P + q]) * es);
                }
        }
        b.bytes[send_buf(r)] = sb;
        b.bytes[recv_buf(P, r)] = rb;
    }
    b.bytes[scratch_buf(P)] = scratch_bytes;
    return b;
}

bool lower(const CollectiveSpec& s, HostProgram& p, std::string& err) {
    p = HostProgram();
    p.P = s.P;
    p.phase_mode = s.phases;
    if (s.coll == COLL_ALLTOALLV) {
        lower_alltoallv(s, p);
        return true;
    }
    if (s.coll == COLL_ALLTOALLV_DYNAMIC) {
        if (s.P > kMaxRanks || s.row_elems == 0) {
            err = "alltoallv_dynamic needs 1..64 ranks and row_elems >= 1";
            return false;
        }
        if (dynamic_tile_bound(s) >= (1ull << 31)) {
            err = "alltoallv_dynamic capacities too large for one exchange";
            return false;
        }
        lower_alltoallv_dynamic(s, p);
        return true;
    }
    int algo = resolve_algo(s);
    if (s.order == ORDER_HALVING && !is_pow2(s.P)) {
        err = "the recursive-halving order needs a power-of-two number of ranks";
        return false;
    }
    if (s.order == ORDER_HALVING && algo != ALGO_RHD && algo != ALGO_DIRECT) {
        err = "the recursive-halving order is produced by the RHD or DIRECT schedules";
        return false;
    }
    if (algo == ALGO_RHD && s.order != ORDER_HALVING && s.coll != COLL_ALLGATHER) {
        err = "the RHD schedule folds in the recursive-halving order (set order = HALVING)";
        return false;
    }
    if (algo == ALGO_RHD && !is_pow2(s.P)) {
        err = "the RHD schedule needs a power-of-two number of ranks";
        return false;
    }
    if (algo == ALGO_TWO_LEVEL && s.order != ORDER_ASCENDING) {
        err = "the two-level schedule has its own grouped order";
        return false;
    }
    if (algo == ALGO_RHD) {
        lower_rhd(s, p);
    } else if (algo == ALGO_TWO_LEVEL) {
        if (s.coll != COLL_ALLREDUCE) {
            err = "the two-level schedule is defined for allreduce only";
            return false;
        }
        if (s.group_size < 1 || s.P % s.group_size != 0) {
            err = "group_size must divide nranks for the two-level schedule";
            return false;
        }
        lower_two_level(s, p);
    } else if (algo == ALGO_RING) {
        lower_ring(s, p);
    } else if (algo == ALGO_DIRECT) {
        lower_direct(s, p);
    } else {
        err = "unknown algorithm";
        return false;
    }
    if (s.requant && s.redop == RO_SUM && (s.dtype == DT_BF16 || s.dtype == DT_FP16))
        for (auto& d : p.descs)
            if (d.op == OP_REDUCE) d.requant = true;
    return true;
}

// ---------------------------------------------------------------------------- fusion
//
// Rule 1 (chain): B = REDUCE(partial, x...) where partial is the scratch output of REDUCE A
//   (its only destination) and B is the only step that reads that value  ->  B = REDUCE(A's
//   sources, x...). The fold is the same sequence of operations on the same values: A's
//   result was never rounded (it is in the accumulation type), B continued from it.
// Rule 2 (groups): E = REDUCE(p_0, ..., p_{G-1}) where every p_g is the scratch output of a
//   flat REDUCE D_g of L sources that only E reads  ->  E = REDUCE(all D_g sources,
//   group = L): fold each run of L into a partial, then fold the partials, as before.
// Rule 3 (forwarding): F = COPY(x -> y...) where x is the value a step E wrote (same
//   location and element count) and F waits for E  ->  E also writes y... . Except when E is a
//   wide reduction (kSplitMinSources or more sources) and the program splits them (by its phase
//   mode and size): then F stays a step of its own, a later phase that copies E's result once
//   it is complete, and a second such copy of the same value joins the first (F also writes
//   its destinations). Measured on the two-level all-reduce P = 64 x 32 MiB bf16: one step of
//   64 sources and 64 destinations 860 us; 64 sources to one destination, then one source to 63
//   destinations in a second launch, about 770 us.
// Rule 4 (trees): E = REDUCE(a, b) where a and b are the private partials of two binary-tree
//   reductions over equally many sources  ->  E = binary tree over both source lists. This
//   is what a recursive-halving level does; the tree, and so every operation, is unchanged.
// Steps merge only if they share the operator and the re-quantisation rule.
//
// Values are tracked by version: the producer of a source is the last step, in program
// order, that wrote exactly that location. Merged steps forward to the step that absorbed
// them, so later lookups and dependencies resolve to the surviving step.
void fuse(HostProgram& p) {
    const uint32_t scratch = scratch_buf(p.P);
    const uint32_t D = (uint32_t)p.descs.size();
    std::vector<uint32_t> fwd(D);
    for (uint32_t i = 0; i < D; ++i) fwd[i] = i;
    // whether the forwarding copies of wide reductions stay separate steps (by the bytes the
    // reductions read from the send buffers)
    uint64_t reduce_bytes = 0;
    for (const auto& d : p.descs)
        if (d.op == OP_REDUCE)
            for (const Operand& o : d.srcs)
                if (o.buf < (uint32_t)p.P) reduce_bytes += d.nelem * dtype_size(o.dtype);
    const bool split = p.phase_mode == PHASE_LEVELS || (p.phase_mode == PHASE_AUTO && reduce_bytes >= kSplitMinBytes);
    // split copies, by the value they read: a second copy of that value joins the first
    std::unordered_map<OperandKey, uint32_t, OperandKeyHash> split_copy;
    auto find = [&](uint32_t x) {
        while (fwd[x] != x) {
            fwd[x] = fwd[fwd[x]];
            x = fwd[x];
        }
        return x;
    };

    // producer of every source operand, and how many sources read each written value
    std::vector<std::vector<int64_t>> prod(D);
    std::vector<std::vector<uint32_t>> nread(D);
    {
        std::unordered_map<OperandKey, std::pair<uint32_t, uint32_t>, OperandKeyHash> last;
        for (uint32_t i = 0; i < D; ++i) {
            const HostDesc& d = p.descs[i];
            nread[i].assign(d.dsts.size(), 0);
            prod[i].assign(d.srcs.size(), -1);
            for (size_t k = 0; k < d.srcs.size(); ++k) {
                auto it = last.find({d.srcs[k].buf, d.srcs[k].offset});
                if (it == last.end()) continue;
                const HostDesc& w = p.descs[it->second.first];
                if (w.dsts[it->second.second].dtype != d.srcs[k].dtype || w.nelem != d.nelem) continue;
                prod[i][k] = it->second.first;
                nread[it->second.first][it->second.second] += 1;
            }
            for (size_t k = 0; k < d.dsts.size(); ++k) last[{d.dsts[k].buf, d.dsts[k].offset}] = {i, (uint32_t)k};
        }
    }
    auto depends_on = [&](const HostDesc& d, uint32_t target) {
        for (const Dep& e : d.deps)
            if (find(e.desc) == target) return true;
        return false;
    };
    // A is a partial step (scratch output, one destination) whose single value only B reads,
    // with the same operator and rounding rule as B
    auto partial_of = [&](int64_t a, const HostDesc& B) {
        if (a < 0) return false;
        const HostDesc& A = p.descs[a];
        return A.alive && A.op == OP_REDUCE && A.dsts.size() == 1 && A.dsts[0].buf == scratch &&
               A.redop == B.redop && A.requant == B.requant && A.nelem == B.nelem && nread[a][0] == 1 &&
               depends_on(B, (uint32_t)a);
    };
    // ... folded ascending over its list
    auto private_partial = [&](int64_t a, const HostDesc& B) {
        return partial_of(a, B) && p.descs[a].group == 0 && p.descs[a].fold == FOLD_LIST;
    };
    // ... folded as a complete binary tree (a two-source step is one)
    auto tree_partial = [&](int64_t a, const HostDesc& B) {
        if (!partial_of(a, B)) return false;
        const HostDesc& A = p.descs[a];
        const size_t n = A.srcs.size();
        if ((n & (n - 1)) != 0) return false;
        return A.fold == FOLD_PAIRWISE || (n == 2 && A.group == 0);
    };
    auto absorb_deps = [&](HostDesc& into, const HostDesc& from) {
        into.deps.insert(into.deps.end(), from.deps.begin(), from.deps.end());
    };

    for (uint32_t i = 0; i < D; ++i) {
        HostDesc& B = p.descs[i];
        if (!B.alive) continue;
        if (B.op == OP_REDUCE && B.group == 0 && B.fold == FOLD_LIST && !B.srcs.empty()) {
            // Rule 4 (trees): B adds the roots of two equally sized binary trees, each a private
            // partial -> one binary tree over both leaf lists (a recursive-halving level).
            if (B.srcs.size() == 2 && tree_partial(prod[i][0], B) && tree_partial(prod[i][1], B) &&
                p.descs[prod[i][0]].srcs.size() == p.descs[prod[i][1]].srcs.size() &&
                2 * p.descs[prod[i][0]].srcs.size() <= (size_t)kMaxOperands) {
                std::vector<Operand> srcs;
                std::vector<int64_t> sprod;
                for (int k = 0; k < 2; ++k) {
                    uint32_t a = (uint32_t)prod[i][k];
                    HostDesc& A = p.descs[a];
                    srcs.insert(srcs.end(), A.srcs.begin(), A.srcs.end());
                    sprod.insert(sprod.end(), prod[a].begin(), prod[a].end());
                    absorb_deps(B, A);
                    A.alive = false;
                    fwd[a] = i;
                }
                B.srcs = std::move(srcs);
                prod[i] = std::move(sprod);
                B.fold = FOLD_PAIRWISE;
                continue;
            }
            // Rule 2: every source is a private partial of an equally sized flat reduction.
            bool groups = B.srcs.size() >= 2;
            size_t L = 0, total = 0;
            for (size_t k = 0; groups && k < B.srcs.size(); ++k) {
                int64_t a = prod[i][k];
                if (!private_partial(a, B) || (L && p.descs[a].srcs.size() != L)) {
                    groups = false;
                    break;
                }
                L = p.descs[a].srcs.size();
                total += L;
            }
            if (groups && total <= (size_t)kMaxOperands) {
                std::vector<Operand> srcs;
                std::vector<int64_t> sprod;
                size_t G = B.srcs.size();
                for (size_t k = 0; k < G; ++k) {
                    uint32_t a = (uint32_t)prod[i][k];
                    HostDesc& A = p.descs[a];
                    srcs.insert(srcs.end(), A.srcs.begin(), A.srcs.end());
                    sprod.insert(sprod.end(), prod[a].begin(), prod[a].end());
                    absorb_deps(B, A);
                    A.alive = false;
                    fwd[a] = i;
                }
                B.srcs = std::move(srcs);
                prod[i] = std::move(sprod);
                B.group = (G == 1 || L == 1) ? 0 : (uint16_t)L;
                continue;
            }
            // Rule 1: the first source is a private partial.
            int64_t a = prod[i][0];
            if (private_partial(a, B) && p.descs[a].srcs.size() + B.srcs.size() - 1 <= (size_t)kMaxOperands) {
                HostDesc& A = p.descs[a];
                std::vector<Operand> srcs = A.srcs;
                srcs.insert(srcs.end(), B.srcs.begin() + 1, B.srcs.end());
                std::vector<int64_t> sprod = prod[a];
                sprod.insert(sprod.end(), prod[i].begin() + 1, prod[i].end());
                B.srcs = std::move(srcs);
                prod[i] = std::move(sprod);
                absorb_deps(B, A);
                A.alive = false;
                fwd[a] = i;
            }
            continue;
        }
        if (B.op == OP_COPY && B.srcs.size() == 1 && prod[i][0] >= 0) {
            // Rule 3: a forwarding copy of a value becomes more destinations of its producer.
            uint32_t e = find((uint32_t)prod[i][0]);
            HostDesc& E0 = p.descs[e];
            if (!E0.alive || E0.nelem != B.nelem || !depends_on(B, e)) continue;
            if (split && E0.op == OP_REDUCE && E0.srcs.size() >= kSplitMinSources) {
                // the copy of a wide reduction's result stays a step; an earlier copy of the
                // same value that waits only for that reduction takes its destinations
                bool only_e = true;
                for (const Dep& d : B.deps) only_e &= find(d.desc) == e;
                const OperandKey key{B.srcs[0].buf, B.srcs[0].offset};
                auto it = split_copy.find(key);
                if (only_e && it != split_copy.end()) {
                    HostDesc& S = p.descs[it->second];
                    bool s_only_e = true;
                    for (const Dep& d : S.deps) s_only_e &= find(d.desc) == e;
                    if (S.alive && S.nelem == B.nelem && S.srcs[0].dtype == B.srcs[0].dtype && s_only_e &&
                        S.dsts.size() + B.dsts.size() <= (size_t)kMaxOperands) {
                        S.dsts.insert(S.dsts.end(), B.dsts.begin(), B.dsts.end());
                        nread[it->second].resize(S.dsts.size(), 0);
                        B.alive = false;
                        fwd[i] = it->second;
                        continue;
                    }
                }
                if (only_e) split_copy[key] = i;
                continue;
            }
            HostDesc& E = E0;
            if (E.dsts.size() + B.dsts.size() > (size_t)kMaxOperands) continue;
            bool deps_ok = true;
            for (const Dep& d : B.deps) {
                uint32_t t = find(d.desc);
                if (t != e && t > e) deps_ok = false;
            }
            if (!deps_ok) continue;
            E.dsts.insert(E.dsts.end(), B.dsts.begin(), B.dsts.end());
            nread[e].resize(E.dsts.size(), 0);
            for (const Dep& d : B.deps)
                if (find(d.desc) != e) E.deps.push_back(d);
            B.alive = false;
            fwd[i] = e;
        }
    }
    // resolve every dependency to the step that survived
    for (uint32_t i = 0; i < D; ++i) {
        HostDesc& d = p.descs[i];
        if (!d.alive) continue;
        for (Dep& e : d.deps) e.desc = find(e.desc);
        dedupe_deps(d, i);
    }
    p.fused = true;
    // scratch is needed only if some live step still touches it
    bool uses_scratch = false;
    for (const auto& d : p.descs) {
        if (!d.alive) continue;
        for (const Operand& o : d.srcs) uses_scratch |= (o.buf == scratch);
        for (const Operand& o : d.dsts) uses_scratch |= (o.buf == scratch);
    }
    if (!uses_scratch) p.scratch_bytes = 0;
}

// ------------------------------------------------------------------------------ groups
bool merge(std::vector<HostProgram>& parts, const std::vector<CollectiveSpec>& specs, HostProgram& out,
           std::string& err) {
    out = HostProgram();
    const size_t n = parts.size();
    std::vector<uint32_t> buf_base(n), nbuf(n), meta_base(n), aux_base(n);
    std::vector<uint64_t> scratch_base(n), bytes(n);
    uint32_t total = 0, nmeta = 0, naux = 0;
    uint64_t scratch = 0;
    for (size_t k = 0; k < n; ++k) {
        buf_base[k] = total;
        nbuf[k] = 2u * (uint32_t)specs[k].P;
        total += nbuf[k];
        meta_base[k] = nmeta;
        nmeta += parts[k].nmeta;
        aux_base[k] = naux;
        naux += (uint32_t)parts[k].aux.size();
        scratch_base[k] = scratch;
        scratch += (parts[k].scratch_bytes + 255) & ~uint64_t(255);
        for (const auto& d : parts[k].descs)
            if (d.alive) bytes[k] += d.nelem * (d.srcs.size() + d.dsts.size());
    }
    if (total > 2u * (uint32_t)kMaxRanks) {
        err = "a group may name at most 128 rank buffers";
        return false;
    }
    if (nmeta > (uint32_t)kMaxMetaBuffers) {
        err = "a group may hold at most two dynamic calls";
        return false;
    }
    std::vector<size_t> order(n);
    for (size_t k = 0; k < n; ++k) order[k] = k;
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return bytes[a] < bytes[b]; });
    // merged ids: every call's rank buffers, then the one scratch, then every call's metadata
    const uint32_t scratch_id = total;
    out.P = (int)(total / 2);
    auto move_id = [&](size_t k, uint32_t id) -> uint32_t {
        if (id == kNoBuffer) return kNoBuffer;
        if (id < nbuf[k]) return id + buf_base[k];
        if (id == nbuf[k]) return scratch_id;
        return meta_buf(out.P, (int)(meta_base[k] + (id - nbuf[k] - 1)));
    };
    for (size_t k = 0; k < n; ++k) {
        for (DynA2A a : parts[k].aux) {
            a.send0 = move_id(k, a.send0);
            a.recv0 = move_id(k, a.recv0);
            a.counts = move_id(k, a.counts);
            a.sdispls = move_id(k, a.sdispls);
            a.rdispls = move_id(k, a.rdispls);
            a.recvcounts = move_id(k, a.recvcounts);
            out.aux.push_back(a);
        }
    }
    bool fused = true;
    for (size_t k : order) {
        HostProgram& p = parts[k];
        fused &= p.fused;
        std::vector<int64_t> remap(p.descs.size(), -1);
        const uint32_t first = (uint32_t)out.descs.size();
        for (size_t i = 0; i < p.descs.size(); ++i) {
            if (!p.descs[i].alive) continue;
            remap[i] = (int64_t)(first + (out.descs.size() - first));
            HostDesc d = p.descs[i];
            for (auto* list : {&d.srcs, &d.dsts}) {
                for (Operand& o : *list) {
                    if (o.buf == nbuf[k]) o.offset += scratch_base[k];
                    o.buf = move_id(k, o.buf);
                }
            }
            d.aux += aux_base[k];
            out.descs.push_back(std::move(d));
        }
        for (uint32_t i = first; i < out.descs.size(); ++i) {
            for (Dep& e : out.descs[i].deps) {
                if (remap[e.desc] < 0) {
                    err = "dependency on a removed step";
                    return false;
                }
                e.desc = (uint32_t)remap[e.desc];
            }
        }
    }
    out.nmeta = nmeta;
    out.phase_mode = specs[0].phases;
    out.algo = parts[order[0]].algo;
    out.fused = fused;
    out.scratch_bytes = scratch;
    return true;
}

// ---------------------------------------------------------------------------- packing
bool finalize(HostProgram& p, uint32_t tile_bytes, std::string& err) {
    // compact
    std::vector<int64_t> remap(p.descs.size(), -1);
    std::vector<HostDesc> live;
    for (size_t i = 0; i < p.descs.size(); ++i) {
        if (!p.descs[i].alive) continue;
        remap[i] = (int64_t)live.size();
        live.push_back(std::move(p.descs[i]));
    }
    for (size_t i = 0; i < live.size(); ++i) {
        for (Dep& d : live[i].deps) {
            if (remap[d.desc] < 0) {
                err = "dependency on a removed step";
                return false;
            }
            d.desc = (uint32_t)remap[d.desc];
        }
        dedupe_deps(live[i], (uint32_t)i);
    }
    p.descs = std::move(live);

    // Phases. A step's level is 0 without dependencies, else one more than the highest level it
    // waits for. Run level by level, one launch each, every dependency is met by the launch
    // order: the steps are laid out level by level (program order inside a level) and carry no
    // dependencies on the device. Otherwise the whole program is one launch and its
    // dependencies are waited for tile by tile.
    {
        const uint32_t n = (uint32_t)p.descs.size();
        std::vector<uint32_t> level(n, 0);
        uint32_t nlev = 1;
        bool deps_here = false;
        for (uint32_t i = 0; i < n; ++i) {
            for (const Dep& d : p.descs[i].deps) level[i] = std::max(level[i], level[d.desc] + 1);
            deps_here |= !p.descs[i].deps.empty();
            nlev = std::max(nlev, level[i] + 1);
        }
        const bool by_level = deps_here && nlev <= kMaxPhases &&
                              (p.phase_mode == PHASE_LEVELS || (p.phase_mode == PHASE_AUTO && nlev <= kAutoMaxPhases));
        p.desc_phase.assign(n, 0);
        if (by_level) {
            std::vector<uint32_t> order(n);
            for (uint32_t i = 0; i < n; ++i) order[i] = i;
            std::stable_sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) { return level[a] < level[b]; });
            std::vector<HostDesc> sorted;
            sorted.reserve(n);
            for (uint32_t k = 0; k < n; ++k) {
                sorted.push_back(std::move(p.descs[order[k]]));
                sorted.back().deps.clear();  // met by the launch order
                p.desc_phase[k] = level[order[k]];
            }
            p.descs = std::move(sorted);
        }
    }
    const uint32_t nphase = p.descs.empty() ? 1u : p.desc_phase.back() + 1;

    // One tile size for a program with dependencies, so per-tile dependencies line up; without
    // them every step gets the tile size for its own element width (the bf16 rows of a group
    // with int32 ids keep 8 KiB tiles instead of taking the ids' element count).
    uint64_t max_bpe = 1, total_elems = 0;
    std::vector<uint64_t> phase_elems(nphase, 0), phase_wide_copy_bytes(nphase, 0);
    bool any_reduce = false, any_deps = false;
    for (size_t i = 0; i < p.descs.size(); ++i) {
        const auto& d = p.descs[i];
        uint64_t bpe = 0;
        for (const Operand& o : d.srcs) bpe += dtype_size(o.dtype);
        max_bpe = std::max(max_bpe, bpe);
        any_reduce |= d.op == OP_REDUCE;
        any_deps |= !d.deps.empty();
        total_elems += d.nelem;
        phase_elems[p.desc_phase[i]] += d.nelem;
        if (d.op == OP_COPY && d.dsts.size() >= kWideCopyDsts) phase_wide_copy_bytes[p.desc_phase[i]] += d.nelem * bpe;
    }
    uint64_t tb = tile_bytes;
    if (!tb) tb = any_deps ? kDefaultDependentTileBytes : any_reduce ? kDefaultReduceTileBytes : kDefaultCopyTileBytes;
    uint64_t te = (tb / max_bpe) / kWaveStepElems * kWaveStepElems;
    if (!tile_bytes && any_reduce) te = std::max<uint64_t>(te, kMinReduceTileElems);
    if (!tile_bytes && !any_deps)
        te = std::min<uint64_t>(te, total_elems / kSmallTargetTiles / kWaveStepElems * kWaveStepElems);
    if (!tile_bytes && any_deps) {
        auto count_tiles = [&](uint64_t e) {
            uint64_t n = 0;
            for (const auto& d : p.descs) n += std::max<uint64_t>(1, (d.nelem + e - 1) / e);
            return n;
        };
        while (count_tiles(te) < kDependentMinTiles && (te / 2) * max_bpe >= kMinDependentTileBytes &&
               (te / 2) % kWaveStepElems == 0)
            te /= 2;
    }
    te = std::max<uint64_t>(te, kWaveStepElems);
    te = std::min<uint64_t>(te, 1ull << 30);
    p.tile_elems = (uint32_t)te;
    auto step_tile = [&](const HostDesc& h, uint32_t phase) -> uint64_t {
        if (any_deps || tile_bytes) return te;
        uint64_t bpe = 0;
        for (const Operand& o : h.srcs) bpe += dtype_size(o.dtype);
        if (bpe == 0) return te;
        // a copy to many destinations writes its tile to each of them: longer runs per
        // destination, and enough work per tile without cutting it for parallelism
        const bool wide_copy = h.op == OP_COPY && h.dsts.size() >= kWideCopyDsts;
        const uint64_t wide_tb = std::max<uint64_t>(
            kDefaultCopyTileBytes, std::min<uint64_t>(kWideCopyTileBytes, phase_wide_copy_bytes[phase] / kWideCopyTargetTiles));
        uint64_t t = ((wide_copy ? wide_tb : tb) / bpe) / kWaveStepElems * kWaveStepElems;
        if (any_reduce && !wide_copy) t = std::max<uint64_t>(t, kMinReduceTileElems);
        if (!wide_copy)
            t = std::min<uint64_t>(t, phase_elems[phase] / kSmallTargetTiles / kWaveStepElems * kWaveStepElems);
        return std::min<uint64_t>(std::max<uint64_t>(t, kWaveStepElems), 1ull << 30);
    };

    const uint32_t nd = (uint32_t)p.descs.size();
    std::vector<Desc> out(nd);
    std::vector<Operand> ops;
    std::vector<Dep> deps;
    std::vector<uint32_t> tile_owner;
    uint64_t ntiles = 0;
    p.bytes_read = p.bytes_written = 0;
    p.max_srcs = 0;
    p.step_tile_min = p.step_tile_max = 0;
    bool has_deps = false;
    for (uint32_t i = 0; i < nd; ++i) {
        const HostDesc& h = p.descs[i];
        Desc& d = out[i];
        std::memset(&d, 0, sizeof d);
        d.op = h.op;
        d.redop = h.redop;
        d.group = h.group;
        d.nsrc = (uint16_t)h.srcs.size();
        d.ndst = (uint16_t)h.dsts.size();
        d.nelem = h.nelem;
        d.fold = h.fold;
        d.requant = h.requant ? 1u : 0u;
        const uint64_t dte = step_tile(h, p.desc_phase[i]);
        d.tile_elems = (uint32_t)dte;
        if (h.op == OP_COPY || h.op == OP_REDUCE) {
            p.step_tile_min = p.step_tile_min ? std::min<uint32_t>(p.step_tile_min, (uint32_t)dte) : (uint32_t)dte;
            p.step_tile_max = std::max<uint32_t>(p.step_tile_max, (uint32_t)dte);
        }
        d.aux = h.aux;
        uint64_t nt = (h.nelem + dte - 1) / dte;
        if (h.op == OP_DYN_COPY) {
            if (h.aux >= p.aux.size()) {
                err = "dynamic step without its record";
                return false;
            }
            nt = p.aux[h.aux].slots;
        }
        if (nt == 0) nt = 1;
        d.ntiles = (uint32_t)nt;
        d.tile0 = (uint32_t)ntiles;
        ntiles += nt;
        if (ntiles >= (1ull << 31)) {
            err = "program has too many tiles";
            return false;
        }
        d.sig = SIG_INVALID;
        if (h.op == OP_REDUCE && !h.srcs.empty() && !h.dsts.empty()) {
            uint32_t tr = h.srcs.size() > 1 ? h.srcs[1].dtype : h.srcs[0].dtype;
            d.sig = reduce_signature(h.srcs[0].dtype, tr, h.dsts[0].dtype);
        }
        d.src = (uint32_t)ops.size();
        ops.insert(ops.end(), h.srcs.begin(), h.srcs.end());
        d.dst = (uint32_t)ops.size();
        ops.insert(ops.end(), h.dsts.begin(), h.dsts.end());
        d.dep = (uint32_t)deps.size();
        d.ndep = (uint16_t)h.deps.size();
        deps.insert(deps.end(), h.deps.begin(), h.deps.end());
        has_deps |= !h.deps.empty();
        p.max_srcs = std::max<uint32_t>(p.max_srcs, d.nsrc);
        for (const Operand& o : h.srcs) p.bytes_read += h.nelem * dtype_size(o.dtype);
        for (const Operand& o : h.dsts) p.bytes_written += h.nelem * dtype_size(o.dtype);
        for (uint64_t t = 0; t < nt; ++t) tile_owner.push_back(i);
    }
    p.ntiles = (uint32_t)ntiles;
    p.nstate = has_deps ? (uint32_t)(kStateDescBase + nd + ntiles) : kStateDescBase;
    p.flags = has_deps ? (uint32_t)PF_HAS_DEPS : 0u;
    // dependency targets: expected values, state words, signal flags
    for (uint32_t i = 0; i < nd; ++i) {
        for (uint32_t k = 0; k < out[i].ndep; ++k) {
            Dep& e = deps[out[i].dep + k];
            Desc& t = out[e.desc];
            if (e.kind == DEP_ALL) {
                e.expected = t.ntiles;
                e.state = kStateDescBase + e.desc;
                t.flags |= DF_SIGNAL_DESC;
            } else {
                e.expected = 1;
                e.state = kStateDescBase + nd + t.tile0;
                t.flags |= DF_SIGNAL_TILE;
            }
        }
    }
    p.ndeps = (uint32_t)deps.size();
    p.noperands = (uint32_t)ops.size();

    // the leanest executor kernel that covers every step of [d0, d1)
    auto kernel_for = [&](uint32_t d0, uint32_t d1) {
        int kind = kKindCopyOnly;
        bool dynamic = false;
        for (uint32_t i = d0; i < d1; ++i) dynamic |= out[i].op == OP_DYN_COPY;
        for (uint32_t i = d0; i < d1; ++i) {
            if (out[i].op != OP_REDUCE) continue;
            const bool plain = out[i].sig <= SIG_INT32 && out[i].redop == RO_SUM && out[i].fold == FOLD_LIST &&
                               !out[i].requant;
            if (!plain) { kind = kKindGeneric; break; }
            if (kind == kKindCopyOnly) kind = out[i].sig;
            else if (kind != out[i].sig) { kind = kKindGeneric; break; }
        }
        if (dynamic) kind = (kind == kKindCopyOnly) ? kKindDynamic : kKindGeneric;  // the two that run them
        if (kind == kKindCopyOnly) {
            bool aligned = true;
            for (uint32_t i = d0; i < d1; ++i)
                for (uint32_t k = 0; k < (uint32_t)out[i].nsrc + out[i].ndst; ++k) aligned &= (ops[out[i].src + k].offset % 16) == 0;
            if (aligned) kind = kKindCopyAligned;  // the launch falls back if a buffer is not aligned
        }
        return kind;
    };
    p.kind = kernel_for(0, nd);
    p.phase_tile.assign(1, 0);
    p.phase_kind.clear();
    p.phase_xcd.clear();
    for (uint32_t q = 0, i = 0; q < nphase; ++q) {
        const uint32_t d0 = i;
        while (i < nd && p.desc_phase[i] == q) ++i;
        p.phase_kind.push_back(kernel_for(d0, i));
        // A phase of wide reductions reads many buffers per wavefront; numbered XCD by XCD, each
        // XCD works on one stretch of them at a time.
        bool wide = i > d0;
        for (uint32_t k = d0; k < i; ++k) wide &= out[k].op == OP_REDUCE && out[k].nsrc >= kSplitMinSources;
        p.phase_xcd.push_back(wide ? 1 : 0);
        p.phase_tile.push_back(i < nd ? out[i].tile0 : p.ntiles);
    }

    auto align16 = [](uint64_t x) { return (x + 15) & ~uint64_t(15); };
    ProgramHeader hdr;
    std::memset(&hdr, 0, sizeof hdr);
    hdr.magic = kProgramMagic;
    hdr.version = kProgramVersion;
    hdr.ndesc = nd;
    hdr.ntiles = p.ntiles;
    hdr.noperand = p.noperands;
    hdr.ndep = p.ndeps;
    hdr.flags = p.flags;
    hdr.nstate = p.nstate;
    hdr.off_desc = align16(sizeof(ProgramHeader));
    hdr.off_operand = align16(hdr.off_desc + (uint64_t)nd * sizeof(Desc));
    hdr.off_dep = align16(hdr.off_operand + ops.size() * sizeof(Operand));
    hdr.off_tile_desc = align16(hdr.off_dep + deps.size() * sizeof(Dep));
    hdr.off_aux = align16(hdr.off_tile_desc + tile_owner.size() * sizeof(uint32_t));
    hdr.naux = (uint32_t)p.aux.size();
    hdr.nphase = nphase;
    hdr.off_phase = align16(hdr.off_aux + p.aux.size() * sizeof(DynA2A));
    hdr.total_bytes = align16(hdr.off_phase + p.phase_tile.size() * sizeof(uint32_t));
    hdr.scratch_bytes = p.scratch_bytes;
    p.image.assign(hdr.total_bytes, 0);
    std::memcpy(p.image.data(), &hdr, sizeof hdr);
    if (nd) std::memcpy(p.image.data() + hdr.off_desc, out.data(), (size_t)nd * sizeof(Desc));
    if (!ops.empty()) std::memcpy(p.image.data() + hdr.off_operand, ops.data(), ops.size() * sizeof(Operand));
    if (!deps.empty()) std::memcpy(p.image.data() + hdr.off_dep, deps.data(), deps.size() * sizeof(Dep));
    if (!tile_owner.empty())
        std::memcpy(p.image.data() + hdr.off_tile_desc, tile_owner.data(), tile_owner.size() * sizeof(uint32_t));
    if (!p.aux.empty()) std::memcpy(p.image.data() + hdr.off_aux, p.aux.data(), p.aux.size() * sizeof(DynA2A));
    std::memcpy(p.image.data() + hdr.off_phase, p.phase_tile.data(), p.phase_tile.size() * sizeof(uint32_t));
    return true;
}

}  // namespace hccl
