"""The allocation-free FFN entry point (moe_grouped_ffn_persistent_noalloc),
called through the C ABI, against moe_grouped_ffn_persistent on the same
operations: h and y_perm bit for bit (the schedule never changes what a tile
computes), on two calls in a row, the second with fewer tokens, and a third
at the first size again; plus the size check made before any launch."""
import ctypes as C

import numpy as np
import pytest

from _helpers import layer_specs
from workload import custom_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_18002_amd import load_library
    load_library()
    return torch.device("cuda:0")


def _valid_rows(b):
    return (b.row_to_assign >= 0).cpu().numpy()


def _outputs(pipe):
    out = []
    for b in pipe.bufs:
        v = _valid_rows(b)
        out.append((b.h.view(torch.uint8).cpu().numpy()[v], b.y_perm.view(torch.int16).cpu().numpy()[v],
                    b.y.view(torch.int16).cpu().numpy()))
    return out


def _run(pipe, noalloc):
    from paper_2607_18002_amd import ops
    for b in pipe.bufs:
        b.h.zero_()
        b.y_perm.zero_()
    pipe.route()
    pipe.permute()
    if noalloc:
        ops.moe_grouped_ffn_persistent_noalloc(pipe.descs, pipe.cfg, pipe.status)
    else:
        pipe.ffn()
    pipe.combine()
    torch.cuda.synchronize()
    assert pipe.statuses() == (0, 0)
    return _outputs(pipe)


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_noalloc_matches_allocating_entry_point(dev, dtype):
    from paper_2607_18002_amd.pipeline import MoEPipeline
    base = 2 if dtype == "bf16" else 5
    sizes = [(900, 200), (300, 45), (900, 200)]          # tokens (prefill, decode) of calls 1, 2, 3
    for n, (tp, td) in enumerate(sizes):
        print(f"noalloc {dtype} call {n}: {tp} prefill + {td} decode tokens", flush=True)
        cfg = custom_config(base, cfg_id=900 + base + 10 * n, H=512, I=512, prefill_tokens=tp, decode_tokens=td,
                            E_global=64, E_local=16, top_k=4, zipf_s=(1.1,))
        specs, _, _ = layer_specs(cfg, 0, dev, decode={"release_after_ns": 10_000})
        pipe = MoEPipeline(specs, fused_gather=True, masked_decode=True)
        want = _run(pipe, noalloc=False)
        got = _run(pipe, noalloc=True)
        for (h0, y0, t0), (h1, y1, t1) in zip(want, got):
            assert np.array_equal(h0, h1)
            assert np.array_equal(y0, y1)
            assert np.array_equal(t0, t1)


def test_noalloc_rejects_ops_beyond_its_workspace(dev):
    """Ops whose scheduler workspace exceeds the static array are refused on
    the host; nothing is launched and the status word is untouched."""
    from paper_2607_18002_amd import _lib
    from paper_2607_18002_amd.pipeline import MoEPipeline
    cfg = custom_config(2, cfg_id=950, H=256, I=256, prefill_tokens=64, decode_tokens=0, E_global=16, E_local=8,
                        top_k=2)
    specs, _, _ = layer_specs(cfg, 0, dev)
    pipe = MoEPipeline(specs)
    d = _lib.OpDesc.from_buffer_copy(pipe.descs[0])
    d.capacity = 1 << 21                                  # 65536 row tiles of 32 rows: 1 MiB of tables per op
    arr = (_lib.OpDesc * 16)(*([d] * 16))
    lib = _lib.load_library()
    pipe.status.fill_(123)
    rc = lib.moe_grouped_ffn_persistent_noalloc(arr, 16, C.byref(pipe.cfg), pipe.status.data_ptr(), None)
    assert rc == _lib.MOE_ERR_CAPACITY
    assert b"static" in lib.moe_last_error()
    torch.cuda.synchronize()
    assert int(pipe.status.item()) == 123
