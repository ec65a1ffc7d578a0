"""Store-completion ordering of the persistent GRU exchange, checked in the gfx950 code the
library is built from (no GPU needed).

Each step of the persistent recurrence writes h_t to a ring slot with device-scope stores and
then arrives on a grid barrier with an atomic add.  On gfx950 a workgroup barrier does not
wait for other waves' stores, so every wave must wait for its own stores (vmcnt(0)) before
the barrier that precedes the arrival; otherwise a workgroup can announce h_t while parts of
it are still in flight.  This compiles csrc/gru.hip to assembly with the library's own flags
and checks, in every instance of the persistent kernel, that such a wait and a barrier sit
between the last ring-slot store and the first arrival atomic after it."""
import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_1810_09958_amd import build as B  # noqa: E402


def _hipcc():
    try:
        return B.hipcc()
    except RuntimeError:
        return None


@pytest.fixture(scope="module")
def gru_asm(tmp_path_factory):
    cc = _hipcc()
    if cc is None:
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "gru.s"
    cmd = [cc, *B.flags(), "--cuda-device-only", "-S", os.path.join(B.CSRC, "gru.hip"), "-o", str(out)]
    subprocess.run(cmd, check=True, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    return out.read_text()


def _functions(asm, name_part):
    """Map mangled symbol -> its instruction lines, for kernels whose name contains name_part."""
    funcs = {}
    cur = None
    for line in asm.splitlines():
        m = re.match(r"^(_Z\S+):\s*(;.*)?$", line)
        if m:
            cur = m.group(1) if name_part in m.group(1) else None
            if cur:
                funcs[cur] = []
            continue
        if cur is not None:
            funcs[cur].append(line.strip())
            if line.strip().startswith("s_endpgm"):
                cur = None
    return funcs


SLOT_STORE = re.compile(r"^buffer_store_(short|dword)\b.*\bsc1\b")
ARRIVAL = re.compile(r"^global_atomic_add\b")
WAIT_STORES = re.compile(r"^s_waitcnt\b.*\bvmcnt\(0\)")


def test_both_persistent_instances_wait_for_slot_stores_before_arrival(gru_asm):
    funcs = _functions(gru_asm, "gru_recurrent_kernel")
    assert len(funcs) == 2, f"expected the bf16 and fp32 instances, found {list(funcs)}"
    for name, body in funcs.items():
        stores = [i for i, l in enumerate(body) if SLOT_STORE.match(l)]
        assert stores, f"{name}: no device-scope ring-slot store found"
        last = stores[-1]
        arrivals = [i for i, l in enumerate(body) if i > last and ARRIVAL.match(l)]
        assert arrivals, f"{name}: no arrival atomic after the slot store"
        between = body[last + 1: arrivals[0]]
        waits = [i for i, l in enumerate(between) if WAIT_STORES.match(l)]
        assert waits, f"{name}: no vmcnt(0) wait between the slot store and the arrival atomic"
        barriers = [i for i, l in enumerate(between) if l.startswith("s_barrier")]
        assert barriers and barriers[-1] > waits[0], \
            f"{name}: the store wait is not followed by the workgroup barrier before the arrival"
