"""The C-ABI library loads on a machine without a GPU and exports what include/hccl.h declares."""
import ctypes
import os
import re

import pytest

import paper_2608_00358_amd as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hccl.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hccl_[a-z_]+)\s*\(", text)))


def test_header_declarations_match_binding_list():
    assert _declared() == sorted(H.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(H.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), f"{name} missing from libhccl.so"


def test_result_strings_and_config_defaults():
    assert H.hccl_result_string(0) == "hcclSuccess"
    assert H.hccl_result_string(5) == "hcclTimeout"
    cfg = H.hccl_config_init()
    assert cfg.algo == 0 and cfg.fuse == 1 and cfg.chunk_bytes == 0


@pytest.mark.parametrize("n", [0, -1, 65])
def test_comm_create_rejects_bad_rank_counts(n):
    with pytest.raises(H.HcclError) as e:
        H.hccl_comm_create(n, H.NO_DEVICE)
    assert e.value.code == 1


def test_trace_of_a_host_only_communicator_is_empty():
    with H.Comm(4, device=H.NO_DEVICE, trace=1) as c:
        H.hccl_allreduce(c.handle, [1 << 40, 2 << 40, 3 << 40, 4 << 40], [5 << 40, 6 << 40, 7 << 40, 8 << 40], 1000,
                         "fp32")
        rec, khz = c.trace()
    assert rec.shape == (0,)


def test_resident_executor_host_only_rules():
    """A host-only communicator has no device to keep an executor on; stopping one that is not
    running is a no-op, and waiting on one is an error."""
    with H.Comm(4, device=H.NO_DEVICE) as c:
        with pytest.raises(H.HcclError) as e:
            H.hccl_resident_start(c.handle)
        assert e.value.code == 1 and "device" in str(e.value)
        H.hccl_resident_stop(c.handle)
        with pytest.raises(H.HcclError) as e:
            H.hccl_resident_wait(c.handle)
        assert e.value.code == 1
        assert H.hccl_resident_last_seq(c.handle) == 0
