"""The in-place compaction that allocates nothing (static library scratch),
checked through the C ABI against the workspace entry point on the same
inputs: two calls in a row, the second with a smaller input, bit for bit."""

import zlib

import numpy as np
import pytest

import workloads as W
from oracle import prune as OP
from tests.gpu_util import bits, log, raw_bits, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _planes(rng, n_in, hkv, d, hid, prows):
    return (W.payload_bits(rng, (hkv, n_in, d), "bf16"), W.payload_bits(rng, (hkv, n_in, d), "bf16"),
            W.payload_bits(rng, (n_in, hid), "bf16"),
            rng.integers(-2**31, 2**31, size=(prows, n_in), dtype=np.int64).astype(np.int32))


def _dev(cpu):
    k, v, h, p = cpu
    return [to_dev(k, "bf16")], [to_dev(v, "bf16")], to_dev(h, "bf16"), torch.from_numpy(p).cuda()


def test_static_scratch_inplace_matches_workspace_inplace():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08794_amd as A
    rng = np.random.default_rng(zlib.crc32(b"no-alloc"))
    hkv, d, hid, prows = 4, 128, 3584, 3
    # First call larger than the second: the second reuses (and must clear)
    # the counters the first left in the static array.
    for step, (n_in, keep) in enumerate(((65858, 0.72), (9454, 0.35))):
        cpu = _planes(rng, n_in, hkv, d, hid, prows)
        src = np.sort(rng.choice(n_in, int(n_in * keep), replace=False))
        idx = torch.from_numpy(src.astype(np.int32)).cuda()
        log(f"[no-alloc] call {step}: {n_in} -> {src.size} rows")
        ref = _dev(cpu)
        A.apack_compact_kv_inplace(idx, n_in, *ref)
        got = _dev(cpu)
        A.apack_compact_kv_inplace_static(idx, n_in, *got)
        torch.cuda.synchronize()
        for a, b in zip((ref[0][0], ref[1][0], ref[2], ref[3]), (got[0][0], got[1][0], got[2], got[3])):
            assert np.array_equal(bits(a), bits(b))
        # and both are the oracle's gather of the original rows
        np.testing.assert_array_equal(bits(got[0][0])[:, :src.size], OP.compact_rows(cpu[0], src, axis=1))
        np.testing.assert_array_equal(bits(got[2])[:src.size], OP.compact_rows(cpu[2], src, axis=0))
        np.testing.assert_array_equal(got[3].cpu().numpy()[:, :src.size], OP.compact_rows(cpu[3], src, axis=1))


def test_static_scratch_rejects_too_many_rows():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08794_amd as A
    idx = torch.zeros((1 << 20) + 1, dtype=torch.int32, device="cuda")
    x = torch.zeros((1, (1 << 20) + 1, 8), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(A.ApackError, match="static scratch"):
        A.apack_compact_kv_inplace_static(idx, x.shape[1], [x])
