// The validator decides whether two steps are ordered either from bit matrices of the whole
// dependency closure (small programs) or by a backward search over the waits of the later step
// (large ones). This driver compiles collectives with the library's own lowering, fusion and
// finalisation, then validates every program both ways: as compiled, and after mutations that
// take orderings away (one wait dropped; one whole-step wait weakened to a per-tile one, which
// keeps the program well formed only where both steps have the same size). Both forms must give
// the same verdict and the same message. Prints one line per disagreement and a summary; exit
// status 1 on any disagreement or if no mutant was rejected.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <random>
#include <string>

#include "compiler.h"

using namespace hccl;

namespace {

int checked = 0, rejected = 0, mismatched = 0;

void both(const HostProgram& p, const CollectiveSpec& s, const char* what) {
    std::string e_bits, e_search;
    const bool bits = validate(p, s, e_bits, UINT32_MAX);
    const bool search = validate(p, s, e_search, 0);
    ++checked;
    if (!bits) ++rejected;
    if (bits != search || e_bits != e_search) {
        ++mismatched;
        std::printf("MISMATCH %s: bit matrices %d '%s', search %d '%s'\n", what, bits, e_bits.c_str(), search,
                    e_search.c_str());
    }
}

}  // namespace

int main() {
    std::mt19937_64 rng(7);
    const int colls[] = {COLL_ALLREDUCE, COLL_REDUCE_SCATTER, COLL_ALLGATHER};
    const int algos[] = {ALGO_DIRECT, ALGO_RING, ALGO_RHD, ALGO_TWO_LEVEL};
    const int Ps[] = {2, 3, 4, 6, 8};
    const uint64_t counts[] = {1, 777, 5000};
    int programs = 0;
    for (int coll : colls)
        for (int algo : algos)
            for (int P : Ps)
                for (uint64_t count : counts)
                    for (int fuse_on = 0; fuse_on < 2; ++fuse_on)
                        for (int phases : {PHASE_ONE, PHASE_AUTO}) {
                            CollectiveSpec s;
                            s.coll = coll;
                            s.P = P;
                            s.dtype = DT_FP32;
                            s.count = count;
                            s.algo = algo;
                            s.fuse = fuse_on;
                            s.phases = phases;
                            s.chunk_bytes = 512;
                            s.tile_bytes = 256;
                            if (algo == ALGO_RHD) s.order = ORDER_HALVING;
                            if (algo == ALGO_TWO_LEVEL) {
                                if (coll != COLL_ALLREDUCE || P % 2 || P == 2) continue;
                                s.group_size = 2;
                            }
                            HostProgram p;
                            std::string err;
                            if (!lower(s, p, err)) continue;  // unsupported combination
                            if (s.fuse) fuse(p);
                            if (!finalize(p, s.tile_bytes, err)) {
                                std::printf("finalize failed: %s\n", err.c_str());
                                return 1;
                            }
                            ++programs;
                            char what[160];
                            std::snprintf(what, sizeof what, "coll %d algo %d P %d count %llu fuse %d phases %d", coll,
                                          algo, P, (unsigned long long)count, fuse_on, phases);
                            both(p, s, what);
                            // mutants: every dependency of up to 24 sampled steps
                            std::vector<uint32_t> with_deps;
                            for (uint32_t i = 0; i < p.descs.size(); ++i)
                                if (!p.descs[i].deps.empty()) with_deps.push_back(i);
                            std::shuffle(with_deps.begin(), with_deps.end(), rng);
                            if (with_deps.size() > 24) with_deps.resize(24);
                            for (uint32_t i : with_deps) {
                                for (size_t k = 0; k < p.descs[i].deps.size(); ++k) {
                                    HostProgram m = p;
                                    m.descs[i].deps.erase(m.descs[i].deps.begin() + k);
                                    std::snprintf(what, sizeof what, "coll %d algo %d P %d count %llu fuse %d: step %u without wait %zu",
                                                  coll, algo, P, (unsigned long long)count, fuse_on, i, k);
                                    both(m, s, what);
                                    if (p.descs[i].deps[k].kind == DEP_ALL &&
                                        p.descs[p.descs[i].deps[k].desc].nelem == p.descs[i].nelem) {
                                        HostProgram w = p;
                                        w.descs[i].deps[k].kind = DEP_TILE;
                                        std::snprintf(what, sizeof what, "coll %d algo %d P %d count %llu fuse %d: step %u wait %zu per tile",
                                                      coll, algo, P, (unsigned long long)count, fuse_on, i, k);
                                        both(w, s, what);
                                    }
                                }
                            }
                        }
    std::printf("programs %d, validations %d, rejected %d, mismatched %d\n", programs, checked, rejected, mismatched);
    return (mismatched == 0 && rejected > 0 && programs > 0) ? 0 : 1;
}
