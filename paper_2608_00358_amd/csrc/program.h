// program.h -- the descriptor program shared by the host compiler and the device executor.
//
// A program is the single-GPU form of a work packet (paper, Section III-B-2 "Data Path"):
// a topologically ordered list of steps (descriptors, the analogue of WQEs) with explicit
// dependency ids. Descriptors refer to buffers by id, never by address, so a compiled
// program is reused for any buffers of the same shape (work packet caching, Section V-B);
// the addresses arrive in the kernel arguments of each launch.
//
// Buffer ids: 0..P-1 = send buffers, P..2P-1 = receive buffers, 2P = the communicator's
// FP32 scratch, then the device metadata arrays of dynamic collectives (2P+1, ...).
//
// Each descriptor is cut into tiles of `tile_elems` elements; tiles are numbered globally
// in descriptor order. Wavefront w of a grid of W runs tiles w, w + W, ... in order (or, on
// request, takes tiles by atomic ticket). A tile only waits for tiles with lower numbers, so
// the lowest unfinished tile can always run.
//
// A program is run as one or more phases: consecutive ranges of tiles, each its own executor
// launch on the stream, so that everything a phase wrote is visible to the next (the end of a
// kernel is a device-wide release, the start of the next an acquire). A dependency between
// steps of different phases is therefore met by the launch order and is not in the image;
// only dependencies inside one phase are waited for on the device.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace hccl {

constexpr uint32_t kProgramMagic = 0x4C434348u;  // "HCCL"
constexpr uint32_t kProgramVersion = 2;
constexpr uint32_t kMaxPhases = 64;  // launches of one program
constexpr int kMaxOperands = 64;   // sources or destinations of one descriptor (one per lane)
constexpr int kMaxRanks = 64;
constexpr int kMaxMetaBuffers = 8;      // metadata arrays of the dynamic calls of one program
constexpr int kMetaPerDynamicCall = 4;  // counts, send offsets, receive offsets, received counts
constexpr int kMaxBuffers = 2 * kMaxRanks + 1 + kMaxMetaBuffers;
constexpr uint32_t kNoBuffer = 0xFFFFFFFFu;
constexpr int kVecElems = 8;       // elements per lane per vector step
constexpr int kWaveSize = 64;

enum Op : uint8_t {
    OP_COPY = 0,    // byte copy of src[0] to every destination (NMC "A = B")
    OP_REDUCE = 1,  // fold of all sources in list order, rounded once, to every destination
    // (2 is unused: the paper's NOOP WQE, a step that only carries dependencies so that a WQE
    // can wait for several others, is not needed here: every step lists any number of
    // dependency ids itself, so a join is the waiting step's own dependency list)
    // AllToAllvDynamic (device-resident layout): tile k ("slot" k) reads the count matrix from
    // device memory, checks the layout and moves its share of the rows. Names a DynA2A record.
    OP_DYN_COPY = 4,
};

enum DType : uint8_t { DT_BF16 = 0, DT_FP16 = 1, DT_FP32 = 2, DT_INT32 = 3 };
enum RedOp : uint8_t { RO_SUM = 0, RO_MAX = 1, RO_MIN = 2 };

// How a REDUCE folds its source list.
enum Fold : uint32_t {
    FOLD_LIST = 0,      // ascending over the list (grouped when `group` > 0)
    FOLD_PAIRWISE = 1,  // complete binary tree over the list: (s0 s1)(s2 s3)..., then pairs of
                        // those, ...; the list length is a power of two
};

enum DepKind : uint32_t {
    DEP_ALL = 0,   // wait until every tile of the named descriptor has completed
    DEP_TILE = 1,  // wait until the tile with the same index of the named descriptor has completed
};

enum DescFlags : uint8_t {
    DF_SIGNAL_DESC = 1,  // count completed tiles in the descriptor counter (someone waits for DEP_ALL)
    DF_SIGNAL_TILE = 2,  // set the per-tile flag (someone waits for DEP_TILE)
};

enum ProgramFlags : uint32_t {
    PF_HAS_DEPS = 1,     // some descriptor waits; counters must be reset after each launch
};

inline uint32_t dtype_size(uint32_t dt) { return (dt == DT_BF16 || dt == DT_FP16) ? 2u : 4u; }

struct Operand {        // 16 bytes
    uint32_t buf;       // buffer id
    uint32_t dtype;     // element type of this operand
    uint64_t offset;    // byte offset of element 0 of the descriptor in that buffer
};

struct Dep {            // 16 bytes
    uint32_t desc;      // descriptor waited for (lower index than the waiter)
    uint32_t kind;      // DepKind
    uint32_t expected;  // counter value that means "done": ntiles of desc (DEP_ALL) or 1 (DEP_TILE)
    uint32_t state;     // state word: kStateDescBase + desc (DEP_ALL) or the flag of tile 0 of
                        // desc (DEP_TILE; the waiter adds its own tile index)
};

// Element-type signatures a REDUCE may have: (type of source 0, type of the other sources,
// type of the destinations). Chained steps carry FP32 partials next to 16-bit inputs; the
// two-level schedule folds FP32 partials into a 16-bit result.
enum Signature : uint8_t {
    SIG_BF16 = 0, SIG_FP16, SIG_FP32, SIG_INT32,        // (T, T, T)
    SIG_BF16_TO_F32, SIG_F32_BF16_TO_F32, SIG_F32_BF16_TO_BF16, SIG_F32_TO_BF16,
    SIG_FP16_TO_F32, SIG_F32_FP16_TO_F32, SIG_F32_FP16_TO_FP16, SIG_F32_TO_FP16,
    SIG_COUNT,
    SIG_INVALID = 255,
};

// Executor kernel specialisations ("kinds"): a plain signature id for programs whose
// reductions all have that signature and SUM, or one of these.
constexpr int kKindCopyOnly = SIG_COUNT;         // no reductions at all
constexpr int kKindGeneric = SIG_COUNT + 1;      // anything else
constexpr int kKindCopyAligned = SIG_COUNT + 2;  // copies only, every operand 16-byte aligned
constexpr int kKindDynamic = SIG_COUNT + 3;      // copies and AllToAllvDynamic steps
constexpr int kNumKinds = SIG_COUNT + 4;

inline uint8_t reduce_signature(uint32_t t0, uint32_t tr, uint32_t to) {
    if (t0 == tr && tr == to) return (uint8_t)t0;  // DT_* and SIG_* plain ids coincide
    for (uint32_t h = DT_BF16; h <= DT_FP16; ++h) {
        uint8_t base = (h == DT_BF16) ? SIG_BF16_TO_F32 : SIG_FP16_TO_F32;
        if (t0 == h && tr == h && to == DT_FP32) return base;
        if (t0 == DT_FP32 && tr == h && to == DT_FP32) return base + 1;
        if (t0 == DT_FP32 && tr == h && to == h) return base + 2;
        if (t0 == DT_FP32 && tr == DT_FP32 && to == h) return base + 3;
    }
    return SIG_INVALID;
}

struct Desc {           // 64 bytes
    uint8_t op;
    uint8_t redop;
    uint8_t flags;
    uint8_t sig;        // Signature of a REDUCE
    uint16_t nsrc;
    uint16_t ndst;
    uint16_t group;     // fold order: 0 = ascending over all sources; L = ascending inside
                        // each run of L sources into an FP32 partial, then over the partials
    uint16_t ndep;
    uint32_t src;       // index of the first source operand
    uint32_t dst;       // index of the first destination operand
    uint32_t dep;       // index of the first dependency
    uint32_t tile0;     // global number of this descriptor's first tile
    uint32_t ntiles;
    uint32_t tile_elems;
    uint64_t nelem;
    uint32_t fold;      // FOLD_LIST (grouped / flat, per `group`) or FOLD_PAIRWISE
    uint32_t requant;   // 1 = round every partial to the destination type
    uint32_t aux;       // OP_DYN_COPY: index of the DynA2A record
    uint32_t pad1;
};
static_assert(sizeof(Desc) == 64, "descriptor layout");

// Auxiliary record of an AllToAllvDynamic (Section IV-B-2): where its layout is read from.
// Counts and offsets are int64 rows of `row_elems` elements.
struct DynA2A {            // 72 bytes
    uint32_t P;
    uint32_t elem_bytes;
    uint32_t send0;        // buffer id of send buffer 0 (send buffer s is send0 + s)
    uint32_t recv0;        // buffer id of receive buffer 0
    uint32_t counts;       // buffer id of the count matrix, [s*P + d]
    uint32_t sdispls;      // buffer id of explicit send offsets [s*P + d], or kNoBuffer (packed)
    uint32_t rdispls;      // buffer id of explicit receive offsets [d*P + s], or kNoBuffer (packed)
    uint32_t recvcounts;   // buffer id of the received-count output [d*P + s], or kNoBuffer
    uint32_t slots;        // tiles of the step; slot k moves dynamic tiles k, k + slots, k + 2 slots, ...
    uint32_t pad;
    uint64_t row_elems;
    uint64_t send_cap;     // rows per send buffer
    uint64_t recv_cap;     // rows per receive buffer
    uint64_t tile_elems;   // elements per dynamic tile
};
static_assert(sizeof(DynA2A) == 72, "auxiliary record layout");

// Device image: header, then the arrays at the offsets the header records (16-byte aligned).
// An image never changes while a kernel that may read it runs: the executor reads the header,
// the descriptors and the AllToAllvDynamic records through the constant address space, whose
// scalar cache is not kept coherent with writes made during a kernel (each launch starts with
// it invalidated). A launched executor reads only the image it was given; the resident executor,
// which outlives many packets, reads images uploaded before their packets were published, and
// those images are kept until the communicator is destroyed, so no address it has read is
// reused for another image while it runs.
struct ProgramHeader {
    uint32_t magic;
    uint32_t version;
    uint32_t ndesc;
    uint32_t ntiles;
    uint32_t noperand;
    uint32_t ndep;
    uint32_t flags;
    uint32_t nstate;       // u32 words of device state (2 + ndesc + ntiles when PF_HAS_DEPS)
    uint64_t off_desc;
    uint64_t off_operand;
    uint64_t off_dep;
    uint64_t off_tile_desc;  // u32 per tile: the descriptor that owns it
    uint64_t total_bytes;
    uint64_t scratch_bytes;
    uint64_t off_aux;      // DynA2A records
    uint32_t naux;
    uint32_t nphase;       // phases (launches) of the program, 1 .. kMaxPhases
    uint64_t off_phase;    // nphase + 1 u32 tile numbers: phase p runs tiles [t[p], t[p+1])
    uint64_t pad;
};
static_assert(sizeof(ProgramHeader) % 16 == 0, "arrays follow the header 16-byte aligned");

// Device state words: [0] ticket counter, [1] finished-wavefront counter, then one tile
// counter per descriptor, then one flag per tile. All zero between launches.
constexpr uint32_t kStateTicket = 0;
constexpr uint32_t kStateDone = 1;
constexpr uint32_t kStateDescBase = 2;

// Device-side error record (per communicator).
struct ErrorRecord {
    uint32_t code;   // 0 = none, 1 = dependency wait timed out, 2 = a dynamic layout was invalid,
                     // 3 = the trigger word never satisfied its comparison
    uint32_t desc;
    uint32_t tile;
    uint32_t pad;
};

// Per-tile trace record (work-packet counters, Section V-C): wall-clock times (the device's
// constant-rate counter) of one tile, and where it ran.
struct TileStamp {      // 32 bytes
    uint64_t start;     // the wavefront took the tile
    uint32_t ready;     // ticks from start until its dependencies were satisfied
    uint32_t done;      // ticks from start until its data was moved and its signals set
    uint32_t wave;      // executor wavefront that ran it
    uint32_t where;     // XCC id << 24 | shader engine << 16 | CU << 8 | SIMD
    uint64_t pad;
};
static_assert(sizeof(TileStamp) == 32, "trace record layout");

// Kernel arguments of one executor launch.
struct LaunchArgs {
    const uint8_t* prog;     // device image (ProgramHeader first)
    uint32_t* state;         // nstate words
    ErrorRecord* error;
    uint32_t nworkers;       // wavefronts in the grid
    uint32_t dynamic;        // 1 = tiles by atomic ticket; 0 = wavefront w runs tiles w,
                             // w + nworkers, ... (counters used only by dependencies)
    uint64_t timeout_ticks;  // watchdog for one dependency wait, in wall-clock counter ticks
    // Device trigger (Section IV-B-3): no tile starts before (*wait_addr CMP wait_value) holds
    // (wait_addr NULL: start at once). The completion word is set by a kernel of its own.
    const uint64_t* wait_addr;
    uint64_t wait_value;
    uint32_t wait_cmp;       // TriggerCmp
    uint32_t xcd_order;      // 1 = wavefront numbers grouped by XCD (see the kernel), 0 = in block order
    uint32_t tile_begin;     // the tiles of this launch (one phase of the program):
    uint32_t tile_end;       // [tile_begin, tile_end)
    TileStamp* trace;        // one record per tile of the program, or NULL (no trace)
    char* bufs[kMaxBuffers];
};

// Resident executor: work packets handed to an executor that is already running, through a
// ring of slots in coherent pinned host memory (the doorbell). The host fills a slot's
// arguments, then publishes its sequence number; every workgroup polls that number, runs the
// packet, and the last workgroup to finish reports the sequence number back.
constexpr uint32_t kResidentSlots = 64;

constexpr uint64_t kResidentStop = 1ull << 63;  // set in a slot's seq: no packet, the executor ends

// Why a resident executor ended.
enum ResidentExit : uint32_t {
    RESIDENT_EXIT_STOP = 1,        // the host's stop request
    RESIDENT_EXIT_IDLE = 2,        // no packet arrived within the idle limit
    RESIDENT_EXIT_WORKGROUPS = 3,  // the workgroups did not all finish a packet within the watchdog
};

struct ResidentSlot {
    uint64_t seq;      // written last by the host: the packet's sequence number (1, 2, ...),
                       // with kResidentStop set for the stop request (one read gives both)
    uint64_t pad;
    LaunchArgs args;   // nworkers, dynamic and the trigger fields are ignored
};

struct ResidentQueue {
    uint64_t done_seq;   // written by the device: every packet up to this number has completed
    uint32_t error;      // first error code of any completed packet (ErrorRecord codes), sticky
    uint32_t exited;     // written by the device when the executor has stopped taking packets:
                         // why (ResidentExit, never 0)
    uint32_t err_desc;
    uint32_t err_tile;
    uint64_t pad[5];
    ResidentSlot slots[kResidentSlots];
};

// The host writes and the device reads these in place: their layout must not depend on the compiler.
static_assert(sizeof(LaunchArgs) % 8 == 0, "packet arguments are copied in 8-byte words");
static_assert(offsetof(ResidentSlot, args) == 16, "slot header is two words");
static_assert(offsetof(ResidentQueue, slots) == 64, "queue header is one cache line");
static_assert(sizeof(ResidentSlot) % 8 == 0, "slots stay 8-byte aligned");

// Kernel arguments of the resident executor. `ctl` is device memory, zero at launch: word 0
// counts the workgroups that finished the current packet, word 1 is the last packet they all
// finished, word 2 the last packet the relay (the last workgroup) published to the others,
// word 3 its stop flag. `mirror` holds two device copies of packet arguments: packet k uses
// copy k mod 2.
struct ResidentArgs {
    ResidentQueue* q;
    uint32_t* ctl;
    uint64_t* mirror;
    ErrorRecord* error;
    uint64_t timeout_ticks;  // watchdog for one dependency wait or completion wait
    uint64_t idle_ticks;     // the executor ends after this long without a packet
};

enum TriggerCmp : uint32_t { CMP_EQ = 0, CMP_NE = 1, CMP_GE = 2, CMP_GT = 3, CMP_LE = 4, CMP_LT = 5 };

// Kernel arguments of a one-step program launched inline: the step and its operands,
// already resolved to addresses of element 0, travel in the launch packet.
struct InlineArgs {
    uint64_t nelem;
    uint32_t tile_elems;
    uint32_t ntiles;
    uint32_t nworkers;
    uint32_t op;
    uint32_t sig;
    uint32_t redop;
    uint32_t nsrc;
    uint32_t ndst;
    uint32_t group;
    uint32_t es_first;   // element bytes of source 0 (and of a copy)
    uint32_t es_rest;    // element bytes of the other sources
    uint32_t es_out;     // element bytes of the destinations
    uint32_t fold;       // Fold of the step
    uint32_t requant;    // 1 = round every partial to the destination type
    uint64_t src[kMaxOperands];
    uint64_t dst[kMaxOperands];
};

}  // namespace hccl
