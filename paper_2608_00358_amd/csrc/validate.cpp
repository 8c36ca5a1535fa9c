// validate.cpp -- structural checks of a finalized descriptor program (host only).
//
// The paper's compiled model puts the whole dependency structure of a collective in the
// host-generated graph (Section III-B-2: Fence, Sync, WQE Sync, Receive Sync, Send Sync and
// NOOP joins). Here every ordering is an explicit dependency id (a join is a step's list of
// several), so the host can prove, before
// anything runs, that the program is well formed:
//   * every dependency names an earlier step (the program is topologically ordered), and a
//     per-tile dependency joins two steps with the same tiling;
//   * every operand lies inside its buffer;
//   * two steps that touch overlapping bytes, one of them writing, are ordered by the
//     dependency closure (per tile only when both walk the bytes with the same tiling) or by
//     running in different phases (launches), the earlier phase first;
//   * every scratch byte a step reads was written by a step ordered before it;
//   * the steps write exactly the bytes the collective defines as its output (for a dynamic
//     exchange, whose bytes depend on the counts: one dynamic step inside the capacities).
#include <algorithm>
#include <cstdio>
#include <map>

#include "compiler.h"

namespace hccl {

namespace {

struct Access {
    uint64_t lo, hi;
    uint32_t desc;
    uint32_t es;
    bool write;
};

struct Bits {
    uint32_t words = 0;
    std::vector<uint64_t> v;
    void init(uint32_t n, uint32_t bits) {
        words = (bits + 63) / 64;
        v.assign((size_t)n * words, 0);
    }
    uint64_t* row(uint32_t r) { return v.data() + (size_t)r * words; }
    const uint64_t* row(uint32_t r) const { return v.data() + (size_t)r * words; }
    bool test(uint32_t r, uint32_t c) const { return (row(r)[c / 64] >> (c % 64)) & 1; }
    void set(uint32_t r, uint32_t c) { row(r)[c / 64] |= 1ull << (c % 64); }
    void merge(uint32_t into, uint32_t from) {
        uint64_t* a = row(into);
        const uint64_t* b = row(from);
        for (uint32_t i = 0; i < words; ++i) a[i] |= b[i];
    }
};

std::string fmt(const char* f, unsigned long long a = 0, unsigned long long b = 0, unsigned long long c = 0) {
    char buf[256];
    std::snprintf(buf, sizeof buf, f, a, b, c);
    return buf;
}

}  // namespace

bool validate(const HostProgram& p, const CollectiveSpec& spec, std::string& err, uint32_t max_bitset_steps) {
    const int P = p.P;
    const uint32_t D = (uint32_t)p.descs.size();
    const uint32_t nbuf = (uint32_t)(2 * P + 1);
    BufferSizes sizes = buffer_sizes(spec, p.scratch_bytes);
    const uint64_t te = p.tile_elems;

    // ------------------------------------------------------------ per-descriptor shape
    for (uint32_t i = 0; i < D; ++i) {
        const HostDesc& d = p.descs[i];
        if (d.srcs.size() > (size_t)kMaxOperands || d.dsts.size() > (size_t)kMaxOperands) {
            err = fmt("step %llu has more than 64 sources or destinations", i);
            return false;
        }
        if (d.op == OP_DYN_COPY) {
            if (!d.srcs.empty() || !d.dsts.empty()) { err = fmt("dynamic step %llu has operands", i); return false; }
            if (d.aux >= p.aux.size()) { err = fmt("dynamic step %llu names record %llu", i, d.aux); return false; }
            const DynA2A& a = p.aux[d.aux];
            const uint32_t nid = (uint32_t)(2 * P + 1) + p.nmeta;
            auto bad_id = [&](uint32_t id, bool optional) { return id == kNoBuffer ? !optional : id >= nid; };
            if (a.P != (uint32_t)P || a.send0 != send_buf(0) || a.recv0 != recv_buf(P, 0) ||
                bad_id(a.counts, false) || a.counts <= scratch_buf(P) || bad_id(a.sdispls, true) ||
                bad_id(a.rdispls, true) || bad_id(a.recvcounts, true)) {
                err = fmt("dynamic step %llu: its record names the wrong buffers", i);
                return false;
            }
            if (a.slots == 0 || a.tile_elems == 0 || a.tile_elems % (kWaveSize * kVecElems)) {
                err = fmt("dynamic step %llu: bad slots or tile size", i);
                return false;
            }
            if (!d.deps.empty()) { err = fmt("dynamic step %llu waits for another step", i); return false; }
        } else if (d.op == OP_COPY) {
            if (d.srcs.size() != 1 || d.dsts.empty()) { err = fmt("COPY step %llu needs 1 source and >= 1 destination", i); return false; }
            for (const Operand& o : d.dsts)
                if (o.dtype != d.srcs[0].dtype) { err = fmt("COPY step %llu changes the element type", i); return false; }
        } else if (d.op == OP_REDUCE) {
            if (d.srcs.empty() || d.dsts.empty()) { err = fmt("REDUCE step %llu has no source or destination", i); return false; }
            for (size_t k = 2; k < d.srcs.size(); ++k)
                if (d.srcs[k].dtype != d.srcs[1].dtype) { err = fmt("REDUCE step %llu mixes source types", i); return false; }
            for (const Operand& o : d.dsts)
                if (o.dtype != d.dsts[0].dtype) { err = fmt("REDUCE step %llu mixes destination types", i); return false; }
            uint32_t tr = d.srcs.size() > 1 ? d.srcs[1].dtype : d.srcs[0].dtype;
            if (reduce_signature(d.srcs[0].dtype, tr, d.dsts[0].dtype) == SIG_INVALID) {
                err = fmt("REDUCE step %llu has an unsupported type signature", i);
                return false;
            }
            if (d.group && (d.group > d.srcs.size() || d.srcs.size() % d.group)) {
                err = fmt("REDUCE step %llu: group %llu does not split %llu sources", i, d.group, d.srcs.size());
                return false;
            }
            if (d.redop > RO_MIN) { err = fmt("REDUCE step %llu has an unknown operator", i); return false; }
            if (d.fold == FOLD_PAIRWISE) {
                const size_t n = d.srcs.size();
                if (d.group || (n & (n - 1))) {
                    err = fmt("REDUCE step %llu: a binary-tree fold needs a power-of-two source list", i);
                    return false;
                }
                for (size_t k = 1; k < n; ++k)
                    if (d.srcs[k].dtype != d.srcs[0].dtype) {
                        err = fmt("REDUCE step %llu: a binary-tree fold needs one source type", i);
                        return false;
                    }
            } else if (d.fold != FOLD_LIST) {
                err = fmt("REDUCE step %llu has an unknown fold", i);
                return false;
            }
        } else {
            err = fmt("step %llu has an unknown op %llu", i, d.op);
            return false;
        }
        for (int side = 0; side < 2; ++side) {
            for (const Operand& o : side ? d.dsts : d.srcs) {
                uint64_t es = dtype_size(o.dtype);
                if (o.buf >= nbuf) { err = fmt("step %llu names buffer %llu", i, o.buf); return false; }
                if (o.offset % es) { err = fmt("step %llu: misaligned operand offset %llu", i, o.offset); return false; }
                if (o.offset + d.nelem * es > sizes.bytes[o.buf]) {
                    err = fmt("step %llu: operand of buffer %llu ends past its size %llu", i, o.buf, sizes.bytes[o.buf]);
                    return false;
                }
            }
        }
        if (p.desc_phase.size() == D && i > 0 && p.desc_phase[i] < p.desc_phase[i - 1]) {
            err = fmt("step %llu is in an earlier phase than step %llu", i, i - 1);
            return false;
        }
        for (const Dep& e : d.deps) {
            if (e.desc >= i) { err = fmt("step %llu depends on step %llu, which is not earlier", i, e.desc); return false; }
            if (p.desc_phase.size() == D && p.desc_phase[e.desc] != p.desc_phase[i]) {
                err = fmt("step %llu waits on the device for step %llu of another phase", i, e.desc);
                return false;
            }
            if (e.kind == DEP_TILE && p.descs[e.desc].nelem != d.nelem) {
                err = fmt("step %llu waits per tile on step %llu with a different size", i, e.desc);
                return false;
            }
        }
    }

    // ---------------------------------------------------------- dependency closure
    // all[y] has x when every tile of x completes before any tile of y starts; tile[y] has x
    // when tile k of x completes before tile k of y starts (chains of per-tile waits).
    // Up to max_bitset_steps steps both relations are D x D bit matrices (144 MB at 24 000).
    // Beyond that a pair is decided by a backward search from the later step over its waits: a
    // path of per-tile waits alone puts x in tile[y], a path with at least one whole-step wait
    // puts it in all[y]; the search visits only steps after x, since every wait names an
    // earlier step.
    bool any_deps = false;
    for (const auto& d : p.descs) any_deps |= !d.deps.empty();
    const bool closure = any_deps && D <= max_bitset_steps;
    Bits all, tile;
    std::vector<uint32_t> seen;  // search stamp of (step, whether a whole-step wait was crossed)
    uint32_t stamp = 0;
    std::vector<std::pair<uint32_t, bool>> todo;
    auto search = [&](uint32_t from, uint32_t x, bool& via_all, bool& via_tile) {
        if (seen.empty()) seen.assign((size_t)2 * D, 0);
        ++stamp;
        todo.assign(1, {from, false});
        while (!todo.empty() && !via_all) {
            const auto [y, crossed] = todo.back();
            todo.pop_back();
            for (const Dep& e : p.descs[y].deps) {
                const bool c = crossed || e.kind == DEP_ALL;
                if (e.desc == x) {
                    (c ? via_all : via_tile) = true;
                } else if (e.desc > x && seen[(size_t)2 * e.desc + c] != stamp) {
                    seen[(size_t)2 * e.desc + c] = stamp;
                    todo.push_back({e.desc, c});
                }
            }
        }
    };
    if (closure) {
        all.init(D, D);
        tile.init(D, D);
        for (uint32_t y = 0; y < D; ++y) {
            for (const Dep& e : p.descs[y].deps) {
                if (e.kind == DEP_ALL) {
                    all.set(y, e.desc);
                    all.merge(y, e.desc);
                    // anything ordered per tile before x is complete when all of x is
                    all.merge(y, e.desc);
                    const uint64_t* t = tile.row(e.desc);
                    uint64_t* a = all.row(y);
                    for (uint32_t w = 0; w < all.words; ++w) a[w] |= t[w];
                } else {
                    tile.set(y, e.desc);
                    tile.merge(y, e.desc);
                    all.merge(y, e.desc);
                }
            }
        }
    }
    // steps of an earlier phase (launch) complete before any step of a later one starts
    const bool phased = p.desc_phase.size() == D;
    auto ordered = [&](const Access& a, const Access& b) {
        // a.desc < b.desc
        if (phased && p.desc_phase[a.desc] < p.desc_phase[b.desc]) return true;
        if (!any_deps) return false;
        bool via_all, via_tile;
        if (closure) {
            via_all = all.test(b.desc, a.desc);
            via_tile = tile.test(b.desc, a.desc);
        } else {
            via_all = via_tile = false;
            search(b.desc, a.desc, via_all, via_tile);
        }
        // per-tile order is enough when both walk identical bytes with the same tiling
        return via_all || (via_tile && a.lo == b.lo && a.es == b.es && a.es != 0);
    };

    // ------------------------------------------------------------------ races
    auto memory_object = [&](uint32_t buf) -> uint32_t {
        if (spec.in_place && buf >= (uint32_t)P && buf < (uint32_t)(2 * P)) return buf - (uint32_t)P;
        return buf;
    };
    std::vector<std::vector<Access>> acc(nbuf);
    for (uint32_t i = 0; i < D; ++i) {
        const HostDesc& d = p.descs[i];
        if (d.op == OP_DYN_COPY) {
            // it may read any send byte and write any receive byte inside the capacities
            // (es = 0: no per-tile identity with another step)
            const DynA2A& a = p.aux[d.aux];
            const uint64_t sb = a.send_cap * a.row_elems * a.elem_bytes;
            const uint64_t rb = a.recv_cap * a.row_elems * a.elem_bytes;
            for (int r = 0; r < P; ++r) {
                if (sb) acc[memory_object(send_buf(r))].push_back(Access{0, sb, i, 0, false});
                if (rb) acc[memory_object(recv_buf(P, r))].push_back(Access{0, rb, i, 0, true});
            }
            continue;
        }
        for (int side = 0; side < 2; ++side) {
            for (const Operand& o : side ? d.dsts : d.srcs) {
                uint64_t es = dtype_size(o.dtype);
                Access a{o.offset, o.offset + d.nelem * es, i, (uint32_t)es, side == 1};
                if (a.hi > a.lo) acc[memory_object(o.buf)].push_back(a);
            }
        }
    }
    for (uint32_t b = 0; b < nbuf; ++b) {
        auto& v = acc[b];
        std::sort(v.begin(), v.end(), [](const Access& x, const Access& y) { return x.lo < y.lo; });
        std::vector<Access> active;
        for (const Access& a : v) {
            active.erase(std::remove_if(active.begin(), active.end(), [&](const Access& x) { return x.hi <= a.lo; }),
                         active.end());
            for (const Access& x : active) {
                if (!(x.write || a.write)) continue;
                if (x.desc == a.desc) {
                    // one step may read and write the same elements (A = A + B) but nothing else
                    if (x.lo == a.lo && x.es == a.es && x.es && x.write != a.write) continue;
                    err = fmt("step %llu touches overlapping bytes of buffer %llu at two positions", a.desc, b);
                    return false;
                }
                const Access& first = x.desc < a.desc ? x : a;
                const Access& second = x.desc < a.desc ? a : x;
                if (!ordered(first, second)) {
                    err = fmt("steps %llu and %llu race on buffer %llu", first.desc, second.desc, b);
                    return false;
                }
            }
            active.push_back(a);
        }
    }

    // -------------------------------------------------- scratch reads follow writes
    const uint32_t sb = scratch_buf(P);
    for (const Access& r : acc[sb]) {
        if (r.write) continue;
        std::vector<std::pair<uint64_t, uint64_t>> cover;
        for (const Access& w : acc[sb]) {
            if (!w.write || w.desc >= r.desc || w.hi <= r.lo || w.lo >= r.hi) continue;
            if (ordered(w, r)) cover.push_back({w.lo, w.hi});
        }
        std::sort(cover.begin(), cover.end());
        uint64_t at = r.lo;
        for (auto& c : cover) {
            if (c.first > at) break;
            at = std::max(at, c.second);
        }
        if (at < r.hi) {
            err = fmt("step %llu reads scratch bytes no earlier ordered step wrote (from %llu)", r.desc, at);
            return false;
        }
    }

    // ----------------------------------------------------------------- coverage
    if (spec.coll == COLL_ALLTOALLV_DYNAMIC) {
        // the bytes written depend on the counts: require the one dynamic step
        if (D != 1 || p.descs[0].op != OP_DYN_COPY) {
            err = "a dynamic exchange is one dynamic step";
            return false;
        }
        return true;
    }
    for (int r = 0; r < P; ++r) {
        uint32_t rb = recv_buf(P, r);
        std::vector<std::pair<uint64_t, uint64_t>> want;
        if (spec.coll == COLL_ALLTOALLV) {
            const uint64_t es = dtype_size(spec.dtype);
            for (int s = 0; s < P; ++s) {
                uint64_t n = spec.recvcounts[(size_t)r * P + s];
                uint64_t o = spec.rdispls[(size_t)r * P + s] * es;
                if (n) want.push_back({o, o + n * es});
            }
        } else if (sizes.bytes[rb]) {
            want.push_back({0, sizes.bytes[rb]});
        }
        std::vector<std::pair<uint64_t, uint64_t>> got;
        for (uint32_t i = 0; i < D; ++i)
            for (const Operand& o : p.descs[i].dsts)
                if (o.buf == rb)
                    got.push_back({o.offset, o.offset + p.descs[i].nelem * dtype_size(o.dtype)});
        auto merge = [](std::vector<std::pair<uint64_t, uint64_t>> v) {
            std::sort(v.begin(), v.end());
            std::vector<std::pair<uint64_t, uint64_t>> out;
            for (auto& x : v) {
                if (x.second <= x.first) continue;
                if (!out.empty() && x.first <= out.back().second) out.back().second = std::max(out.back().second, x.second);
                else out.push_back(x);
            }
            return out;
        };
        if (merge(want) != merge(got)) {
            err = fmt("the steps do not write exactly the output bytes of rank %llu", r);
            return false;
        }
        uint64_t wsum = 0, gsum = 0;
        for (auto& x : merge(want)) wsum += x.second - x.first;
        for (auto& x : got) gsum += x.second - x.first;
        if (wsum != gsum) {
            err = fmt("some output bytes of rank %llu are written more than once", r);
            return false;
        }
    }
    (void)te;
    return true;
}

}  // namespace hccl
