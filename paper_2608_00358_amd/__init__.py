"""HCCL copy/reduce collectives for MI355X (gfx950).

The P ranks of a collective are P buffers in one GPU's HBM. The C library (libhccl.so,
declared in include/hccl.h) lowers each collective into a descriptor program on the host
and runs it with one persistent HIP executor kernel; this package is its ctypes binding.
"""
from .hccl import (  # noqa: F401
    ALGOS, DTYPES, EXPORTS, LIB_PATH, MAX_RANKS, NO_DEVICE, OPS, Comm, HcclError,
    hccl_allgather, hccl_allreduce, hccl_allreduce_noalloc, hccl_alltoallv, hccl_alltoallv_dynamic, hccl_comm_create, hccl_comm_destroy,
    hccl_comm_last_program, hccl_comm_set_config, hccl_comm_program_image, hccl_comm_trace, hccl_config_init, hccl_get_async_error,
    hccl_get_last_error, hccl_group_end, hccl_group_start, hccl_reduce_scatter, hccl_result_string,
    hccl_resident_last_seq, hccl_resident_start, hccl_resident_stop, hccl_resident_wait, hccl_set_trigger, load,
)
