"""Config 4 at full size, in the launch configuration the benchmark times.

The 5-minute 7B clip (7500 audio + 600x144 visual + 128 text tokens, 28 Q /
4 KV heads, head dim 128, hidden 3584): prune steps at layers 14, 18 and 22
keep 0.7, 0.5 and 0.3 of the original audio and visual counts (Algorithm 1,
loop over layers; Eq. 5-6 per modality), each followed by the compaction of
all 28 layers' K/V, the hidden states and the position ids.

Checked against the fp64 oracle, step by step on the rows that survive:
  * kept rows: every index, bit-exact;
  * scores: every candidate within 2e-3 relative;
  * compacted tensors: every row of every plane (28 layers x K and V, the
    hidden states and the position ids), bit-exact against the generator's
    bits at the oracle's kept rows, one plane at a time on the host.
The in-place compaction runs the same three steps on a second copy of the
cache, checked the same way, plus every row past n_out, which must keep its
previous contents.
"""

import numpy as np
import pytest

import workloads as W
from oracle import prune as OP, widen
from tests.gpu_util import bits, log, raw_bits, score_tol, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def cfg4():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08794_amd as A
    A.library()
    log("[cfg4] generating the 5-minute 7B workload with its 28-layer cache")
    pc = W.progressive_case()
    seq = pc.seq()
    n_a, n_v = pc.n_audio, pc.n_visual
    spans, n = list(seq.spans), seq.n_tokens
    rows = np.arange(n)
    steps = []
    for i, (layer, keep) in enumerate(zip(pc.prune_layers, pc.keeps)):
        s = W.PruneSeq(0, n, spans, 0, pc.q_len, (keep, keep), (n_a, n_v))
        k = widen(pc.cache.k_layers[layer], "bf16")[:, rows]
        r = OP.prune_sequence(widen(pc.queries[i], "bf16"), k, s.tags(), s.keep, s.keep_basis)
        del k
        assert r["margin"] >= 1e-2, r["margin"]
        steps.append(dict(seq=s, layer=layer, n_in=n, kept=r["kept"], scores=r["scores"],
                          rows_before=rows, rows_after=rows[r["kept"]]))
        log(f"[cfg4] oracle step {i}: layer {layer}, {n} -> {r['kept'].size} rows, margin {r['margin']:.3g}")
        ka, kv = r["k"]["audio"], r["k"]["visual"]
        spans, n, rows = [(0, ka, W.AUDIO), (ka, kv, W.VISUAL)], r["kept"].size, rows[r["kept"]]
    return pc, steps


def _check_rows(pc, kk, vv, hh, pp, lo, hi, orig_rows):
    """Rows [lo, hi) of every device plane hold the original rows
    `orig_rows` (hi - lo of them), compared plane by plane."""
    for l in range(len(kk)):
        for name, dev, src in (("K", kk, pc.cache.k_layers), ("V", vv, pc.cache.v_layers)):
            got = bits(dev[l][:, lo:hi])
            want = raw_bits(src[l], "bf16")[:, orig_rows]
            assert np.array_equal(got, want), f"{name} layer {l}: {int(np.sum(np.any(got != want, axis=2)))} rows differ"
    assert np.array_equal(bits(hh[lo:hi]), raw_bits(pc.cache.hidden, "bf16")[orig_rows]), "hidden states"
    assert np.array_equal(pp[:, lo:hi].cpu().numpy(), pc.cache.pos[:, orig_rows]), "positions"


def _check_prune(st, scores, kept):
    np.testing.assert_array_equal(kept.cpu().numpy().astype(np.int64), st["kept"])
    got, want = scores.cpu().numpy(), st["scores"]
    tags = st["seq"].tags()
    assert np.all(got[tags == 0] == 0.0)
    c = tags != 0
    rel = np.abs(got[c] - want[c]) / np.abs(want[c])
    assert rel.max() <= score_tol("bf16"), rel.max()


def test_cfg4_full_size_prune_and_compact(cfg4):
    """Three steps back to back on one stream, as the benchmark runs them,
    each step writing its own output cache."""
    import paper_2608_08794_amd as A
    pc, steps = cfg4
    kk = [to_dev(x, "bf16") for x in pc.cache.k_layers]
    vv = [to_dev(x, "bf16") for x in pc.cache.v_layers]
    hh = to_dev(pc.cache.hidden, "bf16")
    pp = torch.from_numpy(pc.cache.pos).cuda()
    out = []
    for i, st in enumerate(steps):
        n_kept, ws_bytes = A.apack_prune_layer_query([st["seq"]], pc.hq, pc.hkv, pc.d)
        m = n_kept[0]
        assert m == st["kept"].size
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        scores = torch.empty(st["n_in"], dtype=torch.float32, device="cuda")
        kept = torch.empty(m, dtype=torch.int32, device="cuda")
        A.apack_prune_layer(to_dev(pc.queries[i], "bf16"), kk[st["layer"]], [st["seq"]], scores=scores,
                            kept_rows=kept, workspace=ws)
        ko = [torch.empty((pc.hkv, m, pc.d), dtype=torch.bfloat16, device="cuda") for _ in kk]
        vo = [torch.empty_like(x) for x in ko]
        ho = torch.empty((m, pc.hidden_dim), dtype=torch.bfloat16, device="cuda")
        po = torch.empty((3, m), dtype=torch.int32, device="cuda")
        A.apack_compact_kv(kept, st["n_in"], kk, vv, ko, vo, hh, ho, pp, po)
        out.append((scores, kept, ko, vo, ho, po))
        kk, vv, hh, pp = ko, vo, ho, po
    torch.cuda.synchronize()
    for i, (st, (scores, kept, ko, vo, ho, po)) in enumerate(zip(steps, out)):
        log(f"[cfg4] checking step {i}: {st['n_in']} -> {kept.numel()} rows")
        _check_prune(st, scores, kept)
        _check_rows(pc, ko, vo, ho, po, 0, kept.numel(), st["rows_after"])


def test_cfg4_full_size_in_place(cfg4):
    """The same three steps compacting one cache in place; after each step
    rows [0, n_out) hold the kept rows and rows [n_out, n_in) are as they
    were."""
    import paper_2608_08794_amd as A
    pc, steps = cfg4
    kk = [to_dev(x, "bf16") for x in pc.cache.k_layers]
    vv = [to_dev(x, "bf16") for x in pc.cache.v_layers]
    hh = to_dev(pc.cache.hidden, "bf16")
    pp = torch.from_numpy(pc.cache.pos).cuda()
    ws = torch.empty(A.apack_compact_kv_inplace_workspace(steps[0]["kept"].size), dtype=torch.uint8, device="cuda")
    for i, st in enumerate(steps):
        n = st["n_in"]
        view = ([x[:, :n] for x in kk], [x[:, :n] for x in vv], hh[:n], pp[:, :n])
        scores, kept, n_kept = A.apack_prune_layer(to_dev(pc.queries[i], "bf16"), view[0][st["layer"]], [st["seq"]])
        A.apack_compact_kv_inplace(kept, n, *view, workspace=ws)
        torch.cuda.synchronize()
        log(f"[cfg4 in place] checking step {i}: {n} -> {kept.numel()} rows")
        _check_prune(st, scores, kept)
        m = kept.numel()
        _check_rows(pc, kk, vv, hh, pp, 0, m, st["rows_after"])
        _check_rows(pc, kk, vv, hh, pp, m, n, st["rows_before"][m:n])
