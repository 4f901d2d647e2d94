"""The read-ceiling probe library: exports, host-side argument checks, and
(on the GPU) that it reads every byte of the buffer exactly once."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_26004_amd import probe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "asymspec_probe.h")


def test_probe_exports_header_symbols():
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(asymspec_[a-z_]+)\s*\(", src)))
    assert names == ["asymspec_probe_clock", "asymspec_probe_read"]
    lib = probe.load_library()
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("src,nbytes,out,nblocks", [
    (0, 1024, 4096, 4),                 # null source
    (4096, 1024, 0, 4),                 # null output
    (4096, 0, 8192, 4),                 # empty buffer
    (4096, 1000, 8192, 4),              # not a multiple of 16
    (4096, (1 << 40) + 16, 8192, 4),    # beyond the stated maximum
    (4096, 1024, 8192, 0),              # no workgroups
    (4096, 1024, 8192, (1 << 20) + 1),  # too many workgroups
    (4104, 1024, 8192, 4),              # source not 16-byte aligned
    (4096, 1024, 8194, 4),              # output not 4-byte aligned
])
def test_probe_rejects_bad_arguments_on_host(src, nbytes, out, nblocks):
    """Every invalid argument is refused before any device work (the
    pointers are never dereferenced: nothing is launched)."""
    st = probe.load_library().asymspec_probe_read(
        ctypes.c_void_p(src), nbytes, ctypes.c_void_p(out), nblocks, None)
    assert st == probe.E_ARG


@pytest.mark.parametrize("out,nblocks,ticks", [
    (0, 4, 100),                          # null output
    (4098, 4, 100),                       # output not 4-byte aligned
    (4096, 0, 100),                       # no workgroups
    (4096, 4097, 100),                    # too many workgroups
    (4096, 4, 0),                         # no wait
    (4096, 4, 1000001),                   # wait beyond the stated maximum
])
def test_clock_probe_rejects_bad_arguments_on_host(out, nblocks, ticks):
    st = probe.load_library().asymspec_probe_clock(ctypes.c_void_p(out), nblocks, ticks, None)
    assert st == probe.E_ARG


@pytest.mark.gpu
def test_clock_probe_reads_a_plausible_clock():
    """The sampled core clock lies between 100 MHz and the part's 2.4 GHz
    peak (with a margin for the counters' granularity)."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    c = probe.clock_mhz(torch.device("cuda"), nblocks=64, ticks=1000)
    print(f"[clock] {c}")
    assert 100.0 < c["min"] <= c["max"] < 2600.0


@pytest.mark.gpu
@pytest.mark.parametrize("nwords,nblocks", [(4, 1), (4 * 12345, 7), (1 << 22, 4096), ((1 << 22) + 4 * 77, 16384)])
def test_probe_reads_every_word(nwords, nblocks):
    """XOR over the per-workgroup results equals the XOR of every 32-bit
    word of the buffer: each 16-byte vector is read once, the ragged end
    included, for grids smaller and larger than the buffer."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    rng = np.random.default_rng(nwords + nblocks)
    host = rng.integers(0, 2**32, size=nwords, dtype=np.uint64).astype(np.uint32)
    dev = torch.device("cuda")
    buf = torch.from_numpy(host.view(np.int32)).to(dev)
    out = torch.full((nblocks,), -1, dtype=torch.int32, device=dev)
    probe.read_xor(buf, out, nblocks)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)
