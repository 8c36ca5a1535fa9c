/*
 * hccl.h -- C ABI of the MI355X copy/reduce collective library.
 *
 * The library follows the compiled communication model of the paper "HCCL: Collective
 * Communication for Meta Training and Inference Accelerators": for every collective the
 * host lowers the call into a complete program of chunked copy / reduce steps with
 * dependency ids (Section III-B-2 "Data Path": work packets, subgraphs, WQEs and their
 * dependency kinds), and one device-resident executor runs that program (Section II-A-2:
 * the message engine's control core unrolls the graph and evaluates dependencies; the
 * near-memory compute unit performs copies and sums with FP32 arithmetic).
 *
 * On one GPU the P ranks of a collective are P buffers in the same HBM: every call takes
 * arrays of P device pointers. Device buffers belong to the caller and must stay valid
 * until the work enqueued on `stream` has completed; the library never frees them. Host
 * arrays (pointer lists, counts, displacements, config) are read during the call only.
 *
 * Every call is enqueue-only: it returns once the work is on `stream` (a hipStream_t
 * passed as void*, NULL = the null stream). Errors are reported by return code; on any
 * error nothing is enqueued. hccl_get_last_error() returns a thread-local description of
 * the last failure. No call aborts or throws across this boundary.
 *
 * Limits: 1 <= nranks <= HCCL_MAX_RANKS. Element counts are in elements of `dtype`.
 * Buffers must be aligned to their element size; 16-byte aligned buffers take the
 * 128-bit vector path, other alignments a vector path with a head and tail of single
 * elements where the destinations allow it, else element by element.
 *
 * Calls on one communicator must not run concurrently from several host threads. Calls
 * may be issued on different streams: the library orders a program's launches by itself.
 *
 * Forward progress: a program whose steps wait for one another (unfused schedules) is launched
 * with a grid sized to the CUs its stream may use. Handed out statically, its tiles need that
 * whole grid resident at once; so while a kernel that waits for something still to come holds
 * CUs of the device (a triggered packet of this process not yet released, a resident executor),
 * such programs take their tiles by atomic ticket, which completes on whatever part of the
 * grid is resident. Kernels of other processes that never finish are not known to the library.
 * While a triggered packet waits, the library also makes no call that could wait for every
 * stream of the device: programs are uploaded on a stream of the communicator that waits for
 * no other, and memory it would free (evicted programs, outgrown scratch) is kept until
 * hccl_comm_destroy.
 *
 * Graph capture: a call (or group) whose program is already compiled enqueues kernel launches
 * only, so it may be made on a stream that is capturing a HIP graph. The first call of a given
 * shape compiles and uploads its program and may grow the communicator's scratch; made under
 * capture it fails with hcclUnsupported and enqueues nothing, so make it once outside the
 * capture first. A graph records the device addresses of the program and the scratch it used;
 * the communicator keeps both allocated until hccl_comm_destroy, after which the graph must
 * not be launched. Launches inside a graph are not ordered by the library against launches of
 * the same program on other streams: the caller orders graph launches against such work.
 */
#ifndef HCCL_H
#define HCCL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HCCL_MAX_RANKS 64
#define HCCL_NO_DEVICE (-1)

typedef enum {
    hcclSuccess = 0,
    hcclInvalidArgument = 1, /* a pointer, size, count, displacement or enum is invalid */
    hcclUnsupported = 2,     /* valid request the library does not implement */
    hcclHipError = 3,        /* a HIP runtime call failed */
    hcclOutOfMemory = 4,     /* device allocation for a program or scratch failed */
    hcclTimeout = 5,         /* a device dependency wait exceeded the watchdog limit */
    hcclInternalError = 6,   /* a compiled program failed validation (library bug) */
} hcclResult_t;

/* Element types of the near-memory compute unit (BF16, FP16, FP32; Section II-A-2),
 * plus INT32 for exact integer reductions and id payloads. */
typedef enum { hcclBf16 = 0, hcclFp16 = 1, hcclFp32 = 2, hcclInt32 = 3 } hcclDataType_t;

/* Reduction operators. SUM is the paper's operator; MAX / MIN are extensions. Floating
 * types are combined in FP32 and rounded once to the buffer type (nearest, ties to even);
 * INT32 SUM wraps modulo 2^32. */
typedef enum { hcclSum = 0, hcclMax = 1, hcclMin = 2 } hcclRedOp_t;

/* Schedules (Section III-B-2 ring AllReduce; Section V-D topology-aware algorithms).
 * All of them fold the contributors of an element in ascending rank order, except
 * TWO_LEVEL, which folds ascending inside each group of `group_size` consecutive ranks
 * into FP32 partials and then folds the partials in ascending group order. */
typedef enum {
    hcclAlgoAuto = 0,     /* TWO_LEVEL when group_size splits nranks, RHD for the HALVING order,
                             else RING */
    hcclAlgoDirect = 1,   /* one step per chunk: read all contributors, write all destinations */
    hcclAlgoRing = 2,     /* ring pipeline: P-1 reduce steps per chunk, then P-1 forwarding hops */
    hcclAlgoTwoLevel = 3, /* group reduce-scatter, inter-group all-reduce of shards, group all-gather */
    hcclAlgoRhd = 4,      /* recursive halving reduce-scatter (+ recursive doubling all-gather);
                             nranks must be a power of two */
} hcclAlgo_t;

/* Order in which the contributors of an element are folded (the result depends on it).
 * ASCENDING: ranks 0, 1, ..., P-1 (TWO_LEVEL: ascending inside each group, then over groups).
 * RING: an element of shard c is folded starting at rank c+1: c+1, c+2, ..., P-1, 0, ..., c,
 *   the order a ring reduce-scatter accumulates it (Section III-B-2 ring AllReduce). For
 *   reduce-scatter, shard c is block c; for all-reduce, element i is in shard i / q with
 *   q = ceil(count / P) rounded up to a multiple of 64.
 * HALVING: the recursive-halving tree: values whose rank differs in bit P/2 are combined first,
 *   then bit P/4, ..., then bit 1 (nranks must be a power of two).
 * With `requantize` set, every partial is rounded to the buffer type as soon as it is formed
 * (the near-memory compute unit re-quantises each result, Section II-A-2); otherwise partials
 * stay FP32 and the result is rounded once. */
typedef enum { hcclOrderAscending = 0, hcclOrderRing = 1, hcclOrderHalving = 2 } hcclOrder_t;

/*
 * Phases (Section III-B-2: a WQE waits for the steps it depends on; Section II-A-2: the control
 * core evaluates those dependencies as it unrolls the work). A compiled program runs as one or
 * more executor launches on the caller's stream, its phases. A dependency between steps of
 * different phases is met by the launch order (a launch ends with its results visible
 * device-wide); only a dependency inside one phase is waited for on the device, tile by tile.
 * AUTO: one launch per dependency level when the program has dependencies and at most 32
 *   levels, otherwise one launch; and when the wide reductions (16 or more sources) of a call
 *   read 256 MiB or more from the send buffers, their results are copied to the other ranks by a
 *   later phase instead of being written to every rank by the reductions themselves.
 * ONE: one launch; dependencies are waited for tile by tile on the device.
 * LEVELS: one launch per dependency level (up to 64), and the copies of every wide reduction's
 *   result run as a later phase.
 * The results are the same in every mode (the same operations in the same order).
 */
typedef enum { hcclPhasesAuto = 0, hcclPhasesOne = 1, hcclPhasesLevels = 2 } hcclPhases_t;

/*
 * Configuration of a communicator (Section V-D: topology-aware algorithm selection, here the
 * schedule, the fold order and the group size of the two-level schedule; Section III-B-2: the
 * work packet's chunking into WQEs, here the chunk and tile sizes). Fields left at zero take the
 * defaults.
 *
 * Two knobs of the paper have no field here. The message engines' cache-partition request
 * bits (Section II-A-3) keep collective buffers from evicting application data; the executor's
 * loads, and its copies' stores, always carry the non-temporal hint instead (the cache policy is
 * an instruction field fixed when the executor is compiled). Per-packet counters (Section V-C)
 * are the `trace` field.
 */
typedef struct {
    int32_t algo;          /* hcclAlgo_t */
    int32_t group_size;    /* ranks per group for TWO_LEVEL; 0 = none */
    uint64_t chunk_bytes;  /* pipeline chunk, bytes of the input type per rank (0 = 1 MiB) */
    int32_t fuse;          /* 1 = fuse chained steps into multi-operand steps (default);
                              0 = run every lowered step as its own dependent descriptor */
    int32_t max_workers;   /* upper bound on executor wavefronts (0 = no bound: one wavefront per
                              tile for a launch whose tiles never wait, else as many as the
                              stream's CUs hold at once) */
    uint32_t tile_bytes;   /* work claimed per ticket, bytes read per tile (0 = default) */
    uint32_t timeout_ms;   /* watchdog for one dependency or trigger wait on the device (0 = 2000) */
    int32_t validate;      /* 1 = run the program validator on every compile */
    int32_t order;         /* hcclOrder_t */
    int32_t requantize;    /* 1 = round every partial to the buffer type */
    int32_t trace;         /* 1 = record times and place of every tile of every launch (hccl_comm_trace) */
    int32_t phases;        /* hcclPhases_t: how a program's steps are spread over launches */
    int32_t reserved;
} hcclConfig_t;

typedef struct hcclComm* hcclComm_t;

/* Fills *cfg with the defaults (automatic schedule, fusion on, every other field zero).
 * hcclInvalidArgument if cfg is NULL. */
hcclResult_t hccl_config_init(hcclConfig_t* cfg);

/*
 * Communicator lifecycle (Section III-B-1 "Control Path": the host creates the resources a
 * collective needs on demand and reuses them; Section V-B: compiled work packets stay in device
 * memory so that a later call only re-enqueues them).
 *
 * Creates a communicator of `nranks` virtual ranks on HIP device `device`. With
 * device == HCCL_NO_DEVICE the communicator is host-only: collective calls validate their
 * arguments and compile (and validate) the program, then return hcclSuccess without
 * touching any buffer or device; hccl_comm_last_program() describes what was compiled.
 * cfg may be NULL (defaults). The communicator owns its program cache, device program
 * copies, dependency counters, FP32 scratch and error word.
 */
hcclResult_t hccl_comm_create(int nranks, int device, const hcclConfig_t* cfg, hcclComm_t* comm);

/* Waits for the communicator's outstanding work, then frees everything it owns. NULL is a no-op.
 * Buffers passed to collectives are the caller's and are not touched. */
hcclResult_t hccl_comm_destroy(hcclComm_t comm);

/* Replaces the configuration used by later calls (cached programs stay valid: the cache is keyed
 * by the whole collective, configuration included). hcclInvalidArgument for a NULL argument. */
hcclResult_t hccl_comm_set_config(hcclComm_t comm, const hcclConfig_t* cfg);

/*
 * The three reduction collectives (Section III-B-2 "Data Path": the ring AllReduce built from
 * receive, NMC sum and send steps; Section II-A-2: the NMC sums BF16 / FP16 / FP32 buffers with
 * FP32 arithmetic and re-quantises the result). sendbufs and recvbufs are arrays of P device
 * pointers (rank r's buffer at index r), aligned to the element size; counts are elements.
 * hcclInvalidArgument for NULL arrays or buffers, misalignment, bad enums or overlapping buffers;
 * hcclUnsupported for a schedule / order combination that does not exist (for example HALVING
 * with a rank count that is not a power of two). Nothing is enqueued on any error.
 *
 * AllReduce: recvbufs[r][i] = R(sendbufs[0][i], ..., sendbufs[P-1][i]) for every rank r
 * and i < count. In place (sendbufs[r] == recvbufs[r] for every r) is allowed; any other
 * overlap between buffers is not.
 */
hcclResult_t hccl_allreduce(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs,
                            size_t count, hcclDataType_t dtype, hcclRedOp_t op, void* stream);

/*
 * Allocation-free AllReduce, for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc. Same result, arguments
 * and argument checks as hccl_allreduce under the communicator's configuration. The call's
 * program image, dependency counters and FP32 partials live in a static workspace of 64 MiB
 * that the library holds on every device it runs on until the process ends; the call makes no
 * hipMalloc, hipFree or other device allocation (its program is compiled, and cached, in host
 * memory). On `stream` it copies the program into the workspace, clears the counters with a
 * fill kernel and launches the executor (a one-step program goes in the launch packet and does
 * not touch the workspace). The communicator must have a device (its error record, allocated
 * by hccl_comm_create, is used); the inputs and outputs are the caller's as usual.
 * Every call on one device shares that workspace and finds it as the last call left it: calls
 * whose work can overlap in time on one GPU (other streams, other communicators) race, and the
 * caller must order them. A call that needs more than the workspace holds (image + counters +
 * partials) fails with hcclInvalidArgument before anything is enqueued. Inside a group, with a
 * pending trigger or while the resident executor runs: hcclUnsupported.
 */
hcclResult_t hccl_allreduce_noalloc(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs,
                                    size_t count, hcclDataType_t dtype, hcclRedOp_t op, void* stream);

/*
 * ReduceScatter (Section III-B-2; the first half of the ring AllReduce): sendbufs[r] holds
 * P * recvcount elements; recvbufs[c][j] =
 * R(sendbufs[0][c*recvcount + j], ..., sendbufs[P-1][c*recvcount + j]). Receive buffers
 * must not overlap any send buffer.
 */
hcclResult_t hccl_reduce_scatter(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs,
                                 size_t recvcount, hcclDataType_t dtype, hcclRedOp_t op, void* stream);

/* AllGather (Section III-B-2, the second half of the ring AllReduce; Section II-A-2: the NMC
 * copy "A = B" doubles as a copy engine): recvbufs[r][q*sendcount + j] = sendbufs[q][j]. A byte
 * copy for every dtype; buffers must not overlap. Errors as for the reductions above. */
hcclResult_t hccl_allgather(hcclComm_t comm, const void* const* sendbufs, void* const* recvbufs,
                            size_t sendcount, hcclDataType_t dtype, void* stream);

/*
 * AllToAllv (Section I: embedding exchange; Section IV-A: spread over parallel engines).
 * For every source s and destination d, n = sendcounts[s*P + d] elements starting at
 * element sdispls[s*P + d] of sendbufs[s] are copied to element rdispls[d*P + s] of
 * recvbufs[d]. Requires recvcounts[d*P + s] == sendcounts[s*P + d] and non-overlapping
 * receive ranges per destination. Receive elements outside every range are untouched.
 * Zero counts are allowed. Count and displacement arrays are host memory, P*P entries.
 */
hcclResult_t hccl_alltoallv(hcclComm_t comm,
                            const void* const* sendbufs, const size_t* sendcounts, const size_t* sdispls,
                            void* const* recvbufs, const size_t* recvcounts, const size_t* rdispls,
                            hcclDataType_t dtype, void* stream);

/*
 * AllToAllvDynamic (Section IV-B-2, device-resident collectives): an AllToAllv whose row
 * counts, and optionally row offsets, are read from device memory when the collective runs,
 * so that a routing kernel earlier on `stream` can write them and nothing on the host waits
 * for it. The program depends only on the capacities and is compiled once; on the device,
 * every slot of it reads the layout, checks it, and moves its share of the rows.
 *
 * All metadata arrays are device memory of P*P int64, 8-byte aligned, counted in rows of
 * `row_elems` elements of `dtype`:
 *   sendcounts[s*P + d]  rows source s sends to destination d (read)
 *   sdispls[s*P + d]     row offset of that range in sendbufs[s] (read); NULL = packed: the
 *                        ranges of one source back to back in ascending destination order
 *   rdispls[d*P + s]     row offset in recvbufs[d] of the rows from s (read); NULL = packed:
 *                        ascending sources back to back from row 0
 *   recvcounts[d*P + s]  = sendcounts[s*P + d] (written; may be NULL)
 * sendbufs[s] holds send_capacity rows and recvbufs[d] recv_capacity rows; the library reads
 * and writes nothing outside them. Send buffers and the read metadata may alias each other;
 * receive buffers and recvcounts alias nothing.
 *
 * A layout with a negative count, a non-empty range outside its buffer, or two overlapping
 * non-empty receive ranges of one destination is rejected on the device: no receive byte is
 * written (recvcounts is still written) and hccl_get_async_error reports hcclInvalidArgument.
 * Until that report is read, later collectives on the communicator do nothing. Ranges of count
 * 0 are never checked. Errors found on the host (arguments) return before anything is enqueued.
 */
hcclResult_t hccl_alltoallv_dynamic(hcclComm_t comm,
                                    const void* const* sendbufs, const int64_t* sendcounts, const int64_t* sdispls,
                                    void* const* recvbufs, int64_t* recvcounts, const int64_t* rdispls,
                                    size_t row_elems, size_t send_capacity, size_t recv_capacity,
                                    hcclDataType_t dtype, void* stream);

/*
 * Groups (one work packet for several collectives, Section III-B-2: a work packet holds
 * several subgraphs). Collectives called on `comm` between hccl_group_start and the
 * matching hccl_group_end are checked when called but only recorded; hccl_group_end
 * compiles them into one program and enqueues it as one executor launch on the stream the
 * calls named (all calls of a group must name the same stream). Groups nest; only the
 * outermost end launches. Buffers of different calls in a group may overlap only where both
 * calls just read them; a group may name at most 128 rank buffers in total (sum of 2 * nranks
 * over its calls) and hold at most two hccl_alltoallv_dynamic calls.
 * On an error in hccl_group_end nothing of the group is enqueued.
 */
hcclResult_t hccl_group_start(hcclComm_t comm);
hcclResult_t hccl_group_end(hcclComm_t comm);

/*
 * Device-triggered collectives (Section IV-B-3). The trigger set here applies to the next work
 * packet the communicator enqueues (one collective called outside a group, or the next
 * outermost hccl_group_end), or rejects, and is then cleared; trigger == NULL clears it.
 *
 * wait_addr (device memory, 8-byte aligned, or NULL): the executor is launched at once and
 *   occupies its CUs, but no step starts until (*wait_addr CMP wait_value) holds, compared as
 *   unsigned 64-bit values. The word is read with system-scope loads, so a kernel on another
 *   stream, a device copy or the host may write it; whatever the writer stored before the word
 *   (inputs, counts) is visible to the collective. Because the waiting executor holds its CUs,
 *   the signalling kernel must find room elsewhere: issue triggered collectives on a CU-masked
 *   stream (hipExtStreamCreateWithCUMask) or cap max_workers. A wait longer than the
 *   communicator's timeout ends the launch with hcclTimeout from hccl_get_async_error; outputs
 *   are then unspecified and the completion word is not written.
 * done_addr (device memory, 8-byte aligned, or NULL): done_value is stored there with a
 *   system-scope release once every step has finished and its results are visible device-wide
 *   (by a one-thread kernel enqueued right behind the executor on the same stream); it is not
 *   written when the launch recorded an error.
 * The two words must not overlap any buffer of the collective.
 */
typedef enum { hcclCmpEq = 0, hcclCmpNe = 1, hcclCmpGe = 2, hcclCmpGt = 3, hcclCmpLe = 4, hcclCmpLt = 5 } hcclCmp_t;

typedef struct {
    const uint64_t* wait_addr;
    uint64_t wait_value;
    int32_t wait_cmp;          /* hcclCmp_t */
    int32_t reserved;
    uint64_t* done_addr;
    uint64_t done_value;
} hcclTrigger_t;

hcclResult_t hccl_set_trigger(hcclComm_t comm, const hcclTrigger_t* trigger);

/* Thread-local text of the last error returned on this thread ("" if none). The string belongs
 * to the library and stays valid until the thread's next failing call. */
const char* hccl_get_last_error(void);

/* Name of a result code (a static string). */
const char* hccl_result_string(hcclResult_t r);

/*
 * Completion errors (Section III-B-2: the message engine reports every work request through a
 * completion queue; Section V-C: completion and event handling on the device side). Work is
 * enqueue-only, so a failure found on the device is kept in the communicator's error record.
 * This call synchronises the communicator's device and reports a device-side failure recorded
 * since the previous call (hcclTimeout when a dependency wait or a trigger wait hit the watchdog,
 * hcclInvalidArgument when a device-resident layout was rejected), then clears it. While a
 * triggered packet waits on the device, this waits for it too.
 */
hcclResult_t hccl_get_async_error(hcclComm_t comm);

/*
 * Resident executor (Section II-A-2: the message engine's control core waits for work packets
 * and runs each as it arrives; Section V-B: once a packet is compiled and cached, handing it
 * over again is the whole per-call cost, which the paper keeps under 10 us).
 *
 * hccl_resident_start launches one executor that stays on the device, on a stream of its own,
 * and takes work packets through a doorbell: a ring of slots in coherent pinned host memory.
 * From then until hccl_resident_stop, every call (or group) on the communicator is handed to it
 * instead of being launched: the call writes the packet's arguments into the next slot and
 * then the slot's sequence number (1, 2, ...), and returns. No kernel is launched per call. A
 * program of several phases (hcclPhases_t) is handed over as one packet per phase, each with
 * its own sequence number, in phase order; hccl_resident_last_seq then names the last.
 *
 *   blocks   workgroups of 4 wavefronts (0 = 32); they must all fit on the device at once,
 *            else hcclInvalidArgument.
 *   idle_ms  the executor ends by itself after this long without a packet (0 = 10 s, at most
 *            10 minutes), so an abandoned executor cannot hold the device.
 *
 * In this mode the `stream` argument of a call is ignored: a packet runs when the executor
 * reaches it, in submission order, one packet at a time. The caller makes the inputs ready
 * (e.g. synchronises the stream that wrote them) before the call, and reads the outputs after
 * hccl_resident_wait has reported the packet complete; outputs are then visible to the host,
 * to copies and to kernels launched afterwards. Submitting more than 64 packets ahead of the
 * executor blocks the call until a slot is free (or fails with hcclTimeout after the
 * communicator's timeout). A packet whose program is not cached is compiled on the host as
 * usual; one that would grow the communicator's scratch, a triggered packet and a call on a
 * capturing stream fail with hcclUnsupported. Programs handed to the executor stay allocated
 * until hccl_comm_destroy. hccl_get_async_error is not available while the executor runs.
 * hipDeviceSynchronize (and anything that waits for every stream of the device) waits for the
 * executor too, which ends only at hccl_resident_stop or its idle limit: synchronise streams.
 */
hcclResult_t hccl_resident_start(hcclComm_t comm, uint32_t blocks, uint32_t idle_ms);

/* Ends the resident executor after the packets already submitted and frees its doorbell;
 * returns once it has left the device. A no-op if it is not running. hccl_comm_destroy stops
 * it too. Afterwards calls are launched on their streams again. */
hcclResult_t hccl_resident_stop(hcclComm_t comm);

/* Waits (on the host, polling pinned memory) until packet `seq` has completed (0 = the last
 * one submitted). Returns hcclTimeout after `timeout_ms` (0 = 2 s) or if the executor ended
 * before the packet ran (idle limit passed), and otherwise the first device error recorded
 * by any completed packet since the last report (hcclInvalidArgument for a rejected
 * device-resident layout, hcclTimeout for a dependency watchdog), which it then clears. */
hcclResult_t hccl_resident_wait(hcclComm_t comm, uint64_t seq, uint32_t timeout_ms);

/* The sequence number of the last packet handed to the resident executor (0 = none). */
hcclResult_t hccl_resident_last_seq(hcclComm_t comm, uint64_t* seq);

/* Description of the most recently compiled or reused program of a communicator. */
typedef struct {
    int32_t collective;          /* 0 allreduce, 1 reduce_scatter, 2 allgather, 3 alltoallv,
                                    4 alltoallv_dynamic, -1 a group */
    int32_t algo;                /* hcclAlgo_t actually lowered */
    int32_t fused;               /* fusion pass applied */
    int32_t cache_hit;           /* 1 if the program came from the cache */
    uint32_t num_descs;          /* descriptors (steps) in the program */
    uint32_t num_tiles;          /* work tickets */
    uint32_t num_deps;           /* dependency edges */
    uint32_t num_operands;       /* operand entries */
    uint32_t workers;            /* wavefronts of the last launch (0 on host-only comms) */
    uint32_t max_srcs;           /* most sources of one step */
    uint32_t inline_launch;      /* 1 if the one-step program travelled in the launch packet */
    uint32_t tickets;            /* 1 if the last launch handed out tiles by atomic ticket (dependent
                                    programs by default; see HCCL_DISPATCH), 0 if statically */
    uint64_t bytes_read;         /* bytes the program's steps read */
    uint64_t bytes_written;      /* bytes the program's steps write */
    uint64_t scratch_bytes;      /* FP32 scratch the program needs */
    uint64_t program_bytes;      /* size of the device copy of the program */
    double compile_us;           /* host time to lower, fuse, validate and pack */
    uint32_t step_tile_min;      /* smallest and largest tile (elements) of the program's copy and */
    uint32_t step_tile_max;      /* reduce steps: steps of different element widths may differ */
    uint32_t num_phases;         /* executor launches per call (see hcclPhases_t) */
    uint32_t reserved;
} hcclProgramInfo_t;

hcclResult_t hccl_comm_last_program(hcclComm_t comm, hcclProgramInfo_t* info);

/*
 * The packed program image of the same program (Section III-B-2: the host builds the complete
 * description of the work packet, its WQEs and their dependency metadata, before the device
 * runs it), exactly as uploaded: a header, then 64-byte steps, 16-byte operands {buffer id,
 * element type, byte offset}, 16-byte dependencies {step, kind, expected count, state word},
 * one owning step per tile and the AllToAllvDynamic records (layout: csrc/program.h). Buffer
 * ids, not addresses, name the operands: send buffers 0..P-1, receive buffers P..2P-1, the
 * scratch 2P (in a group, each call's ids follow the previous calls'). For tools and tests,
 * e.g. an interpreter that runs the steps in any order the dependencies allow. Copies
 * min(capacity, *size) bytes; *size = 0 when the program was evicted or none was compiled.
 */
hcclResult_t hccl_comm_program_image(hcclComm_t comm, void* out, size_t capacity, size_t* size);

/*
 * Per-tile trace (Section V-C: counters on every work packet and subgraph show when each
 * component handled it; the control-core overhead is read off them). With hcclConfig_t.trace
 * set, every launch records, for each tile of its program, the wall-clock time at which an
 * executor wavefront took it, how long its dependency waits lasted, when its data had moved
 * and its signals were set, and where it ran. One-step programs then also run from a device
 * image instead of the launch packet. Launches under graph capture and resident packets are
 * not traced.
 */
typedef struct {
    uint64_t start;     /* wall-clock ticks when a wavefront took the tile */
    uint32_t ready;     /* ticks from start until its dependencies were satisfied */
    uint32_t done;      /* ticks from start until its data had moved and its signals were set */
    uint32_t wave;      /* executor wavefront that ran it */
    uint32_t where;     /* XCC id << 24 | shader engine << 16 | CU << 8 | SIMD */
    uint64_t reserved;
} hcclTileTrace_t;

/* Waits for the device, then copies the records of the last traced launch of `comm` (index =
 * tile number) into out[0 .. min(capacity, *count)). *count = records of that launch (0 if
 * none); *clock_khz (may be NULL) = rate of the wall clock the times use. */
hcclResult_t hccl_comm_trace(hcclComm_t comm, hcclTileTrace_t* out, size_t capacity, size_t* count,
                             uint64_t* clock_khz);

#ifdef __cplusplus
}
#endif
#endif /* HCCL_H */
