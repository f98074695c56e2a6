"""GPU runs of murmur_read_probe, the plain streaming read that bench.py measures the read ceiling with.

The probe computes nothing of the method; these runs check that every configuration of the ceiling sweep
(both load types, every depth and block size, small and large grids, a share that is not a multiple of a
block's loads) launches and ends without a device error, and that the sink (written only when the XOR of
what a workgroup read equals a fixed pattern) stays untouched for data that cannot produce the pattern.
"""
import pytest
import torch

from paper_2606_01483_amd import murmur as M

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    M.lib()
    yield
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0


@pytest.mark.parametrize("nbytes", [16, 4096 * 16 + 48, 3 << 20])
def test_read_probe_configurations(nbytes):
    print(f"\n[case] read probe over {nbytes} bytes", flush=True)
    buf = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")  # XOR of zeros is never the pattern
    sink = torch.zeros(4096, dtype=torch.int32, device="cuda")
    for mode in (M.MURMUR_PROBE_REGISTERS, M.MURMUR_PROBE_LDS):
        for threads in (64, 256, 512, 1024):
            for depth in (1, 2, 4, 8, 16):
                if mode == M.MURMUR_PROBE_LDS and (threads // 64) * depth > 64:
                    continue
                for wg in (1, 256, 4096):
                    M.murmur_read_probe(buf, nbytes, wg, sink, threads, depth, mode)
    torch.cuda.synchronize()
    assert M.murmur_device_error() == 0
    assert int(sink.abs().sum()) == 0
