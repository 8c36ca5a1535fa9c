// compiler.h -- host-side lowering of collectives into descriptor programs.
//
// The host builds the complete description of a collective, dependencies included, before
// anything runs on the device (paper, Section III-B-2 "Data Path"; host-side generation,
// Section V-B). Lowerings emit the schedule step by step (ring reduce chains and forwarding
// hops, two-level group phases); the fusion pass then merges chained steps whose
// intermediate only feeds the next step, which keeps the arithmetic (same operations in
// the same order) and removes the intermediate traffic.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "program.h"

namespace hccl {

enum Collective : int {
    COLL_ALLREDUCE = 0,
    COLL_REDUCE_SCATTER = 1,
    COLL_ALLGATHER = 2,
    COLL_ALLTOALLV = 3,
    COLL_ALLTOALLV_DYNAMIC = 4,  // layout read from device memory when the program runs
};
enum Algo : int { ALGO_AUTO = 0, ALGO_DIRECT = 1, ALGO_RING = 2, ALGO_TWO_LEVEL = 3, ALGO_RHD = 4 };
enum Order : int { ORDER_ASCENDING = 0, ORDER_RING = 1, ORDER_HALVING = 2 };
// How the steps of a program are spread over launches (phases).
//   PHASE_AUTO: one launch per dependency level when the program has dependencies and at most
//     kAutoMaxPhases levels, else one launch; the forwarding copies of wide, large reductions
//     stay separate steps (a second phase) instead of becoming extra destinations.
//   PHASE_ONE: one launch; dependencies are waited for on the device, tile by tile.
//   PHASE_LEVELS: one launch per dependency level, and the forwarding copies of every
//     reduction of kSplitMinSources or more sources stay separate steps.
enum PhaseMode : int { PHASE_AUTO = 0, PHASE_ONE = 1, PHASE_LEVELS = 2 };
constexpr uint32_t kAutoMaxPhases = 32;
constexpr uint32_t kSplitMinSources = 16;
// bytes the wide reductions read from the send buffers, from which PHASE_AUTO splits (the
// two-level all-reduce of 64 ranks, one launch against two: 2 MiB per rank 44-48 / 67 us,
// 4 MiB 98-101 / 90 us, 8 MiB 224 / 203 us, 32 MiB 875-881 / 781-784 us)
constexpr uint64_t kSplitMinBytes = 256ull << 20;

struct CollectiveSpec {
    int coll = COLL_ALLREDUCE;
    int P = 1;
    int dtype = DT_FP32;
    int redop = RO_SUM;
    uint64_t count = 0;          // allreduce: count; reduce_scatter: recvcount; allgather: sendcount
    std::vector<uint64_t> sendcounts, sdispls, recvcounts, rdispls;  // alltoallv, P*P each
    bool in_place = false;       // allreduce with send[r] == recv[r]
    int algo = ALGO_AUTO;
    int group_size = 0;
    uint64_t chunk_bytes = 0;
    bool fuse = true;
    uint32_t tile_bytes = 0;
    int order = ORDER_ASCENDING;
    bool requant = false;        // round every partial to the buffer type
    int phases = PHASE_AUTO;     // PhaseMode
    // alltoallv_dynamic: rows of row_elems elements; buffers hold send_cap / recv_cap rows;
    // which optional metadata arrays the call passes
    uint64_t row_elems = 0, send_cap = 0, recv_cap = 0;
    bool dyn_sdispls = false, dyn_rdispls = false, dyn_recvcounts = false;

    bool operator==(const CollectiveSpec& o) const;
};

struct HostDesc {
    uint8_t op = OP_REDUCE;
    uint8_t redop = RO_SUM;
    uint16_t group = 0;
    uint32_t fold = FOLD_LIST;
    bool requant = false;
    uint64_t nelem = 0;
    std::vector<Operand> srcs;
    std::vector<Operand> dsts;
    std::vector<Dep> deps;
    bool alive = true;
    uint32_t aux = 0;            // OP_DYN_*: index into HostProgram::aux
};

struct HostProgram {
    int P = 0;
    int algo = ALGO_DIRECT;      // schedule actually lowered
    bool fused = false;
    int phase_mode = PHASE_AUTO; // PhaseMode: read by fuse() and finalize()
    uint64_t scratch_bytes = 0;
    std::vector<HostDesc> descs;
    std::vector<DynA2A> aux;     // records of the dynamic steps
    uint32_t nmeta = 0;          // metadata buffer ids in use, from meta_buf(P, 0)

    // filled by finalize()
    uint32_t tile_elems = 0;
    uint32_t step_tile_min = 0;  // smallest and largest per-step tile (elements) of the packed
    uint32_t step_tile_max = 0;  // program; they differ where steps of other widths share it
    uint32_t ntiles = 0;
    uint32_t ndeps = 0;
    uint32_t noperands = 0;
    uint32_t max_srcs = 0;
    uint64_t bytes_read = 0;
    uint64_t bytes_written = 0;
    std::vector<uint8_t> image;  // ProgramHeader + arrays, uploaded to the device as is
    uint32_t nstate = 0;
    uint32_t flags = 0;
    int kind = kKindGeneric;     // executor specialisation that can run every step
    // phases: descriptor p of the packed program belongs to phase desc_phase[p]; phase q runs
    // tiles [phase_tile[q], phase_tile[q + 1]) with kernel phase_kind[q]
    std::vector<uint32_t> desc_phase;
    std::vector<uint32_t> phase_tile;
    std::vector<int> phase_kind;
    std::vector<uint8_t> phase_xcd;  // 1 = the phase's wavefronts are numbered XCD by XCD
    uint32_t nphase() const { return phase_kind.empty() ? 1u : (uint32_t)phase_kind.size(); }
};

// Buffer ids used by lowerings.
inline uint32_t send_buf(int r) { return (uint32_t)r; }
inline uint32_t recv_buf(int P, int r) { return (uint32_t)(P + r); }
inline uint32_t scratch_buf(int P) { return (uint32_t)(2 * P); }
inline uint32_t meta_buf(int P, int i) { return (uint32_t)(2 * P + 1 + i); }
// Metadata arrays of one AllToAllvDynamic call, in buffer-id order from meta_buf(P, 0).
enum MetaSlot : int { META_COUNTS = 0, META_SDISPLS = 1, META_RDISPLS = 2, META_RECVCOUNTS = 3 };

// Byte size of every buffer id a program may touch (for bounds checks and coverage).
struct BufferSizes {
    std::vector<uint64_t> bytes;  // indexed by buffer id, 2P + 1 entries
};
BufferSizes buffer_sizes(const CollectiveSpec& spec, uint64_t scratch_bytes);

inline uint32_t meta_buffers(const CollectiveSpec& s) {
    return s.coll == COLL_ALLTOALLV_DYNAMIC ? (uint32_t)kMetaPerDynamicCall : 0u;
}

// Static tiles of the copy step of an AllToAllvDynamic, and the elements per dynamic tile.
uint32_t dynamic_slots(const CollectiveSpec& s);
uint64_t dynamic_tile_elems(const CollectiveSpec& s);
// Upper bound on the dynamic tiles of any layout that fits the capacities.
uint64_t dynamic_tile_bound(const CollectiveSpec& s);

// Picks the schedule for ALGO_AUTO.
int resolve_algo(const CollectiveSpec& spec);

// Element count of one all-reduce shard: ceil(count / parts) rounded up to 64 elements.
uint64_t shard_size(uint64_t count, int parts);

// Lowers `spec` into `prog` (unfused steps). Returns false and sets err on bad input.
bool lower(const CollectiveSpec& spec, HostProgram& prog, std::string& err);

// Merges chained steps: reduce chains into multi-source reductions, group partial folds into
// grouped reductions, forwarding copies into extra destinations of their producer (except, by
// prog.phase_mode, the copies of wide reductions, which then run as a later phase).
void fuse(HostProgram& prog);

// Merges the (lowered, possibly fused) programs of the collectives of one group into one
// program: call k's buffer ids move up by the ranks of the calls before it (send and
// receive ids of every call stay disjoint), every call's scratch gets its own region of one
// shared scratch, and the calls' steps are laid out smallest call first (the calls are
// independent, so their relative order is free). Returns false if the group is too large.
bool merge(std::vector<HostProgram>& parts, const std::vector<CollectiveSpec>& specs, HostProgram& out,
           std::string& err);

// Removes dead descriptors, assigns phases (prog.phase_mode), renumbers dependencies, cuts
// tiles, sets signal flags, picks each phase's kernel and packs the device image.
// tile_bytes = 0 selects the default.
bool finalize(HostProgram& prog, uint32_t tile_bytes, std::string& err);

// Structural checks of a finalized program: dependency order, operand bounds, per-tile
// dependency shape, data races between steps not ordered by dependencies (with send and
// receive buffers aliased when in_place), and exact coverage of the collective's output.
// Programs of at most max_bitset_steps steps keep the dependency closure as bit matrices, larger
// ones search it pair by pair; both give the same answers.
bool validate(const HostProgram& prog, const CollectiveSpec& spec, std::string& err,
              uint32_t max_bitset_steps = 24000);

}  // namespace hccl
