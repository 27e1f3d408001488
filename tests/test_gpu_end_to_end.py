"""End-to-end launch sequences on the GPU, each stage checked against the oracle.

score_dynamics -> compact (gather of the kept visual embeddings) ->
prune_layer -> compact_kv, enqueued back to back on one stream with no host
synchronisation in between, for
  * a 60 s clip at the 7B shape (1500 audio + 120x144 visual + 64 query rows,
    3584-d embeddings, window 4, R_pre 0.5; prune at keep 0.5 / 0.3 on the
    9454-row sequence), with the gate on and off;
  * a ragged batch of 8 clips of 20-300 s (window 3, R_pre 0.5, keep
    0.5 / 0.3), interleaved 2-second [visual | audio] chunks.
Kept rows and gathered rows are compared bit-exactly; scores and frame
outputs to the stated tolerances.
"""

import numpy as np
import pytest

import workloads as W
from oracle import dynamics as OD, prune as OP, widen
from tests.gpu_util import bits, log, raw_bits, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_08794_amd as A
    A.library()


def _launch(dyn, prune, cache):
    """The whole sequence on one stream; returns device results."""
    import paper_2608_08794_amd as A
    xv, xa, xq = (to_dev(x, "bf16") for x in (dyn.xv, dyn.xa, dyn.xq))
    q, k = to_dev(prune.q, "bf16"), to_dev(prune.k, "bf16")
    v = to_dev(cache.v_layers[0], "bf16")
    hid = to_dev(cache.hidden, "bf16")
    pos = torch.from_numpy(cache.pos).cuda()
    torch.cuda.synchronize()
    sd = A.apack_score_dynamics(xv, xa, xq, dyn.seqs, dyn.params)
    kept_vis = sd["kept"]
    emb = torch.empty((kept_vis.numel(), xv.shape[1]), dtype=xv.dtype, device="cuda")
    A.apack_compact_kv(kept_vis, xv.shape[0], hidden_in=xv, hidden_out=emb)
    scores, kept, n_kept = A.apack_prune_layer(q, k, prune.seqs)
    n_out = sum(n_kept)
    k_out = torch.empty((prune.hkv, n_out, prune.d), dtype=k.dtype, device="cuda")
    v_out = torch.empty_like(k_out)
    h_out = torch.empty((n_out, hid.shape[1]), dtype=hid.dtype, device="cuda")
    p_out = torch.empty((3, n_out), dtype=torch.int32, device="cuda")
    A.apack_compact_kv(kept, k.shape[1], [k], [v], [k_out], [v_out], hid, h_out, pos, p_out)
    torch.cuda.synchronize()
    return dict(dyn=sd, emb=emb, scores=scores, kept=kept, n_kept=n_kept, k_out=k_out, v_out=v_out,
                h_out=h_out, p_out=p_out)


def _check_scorer(dyn, got):
    kept_all = []
    f0 = 0
    for i, s in enumerate(dyn.seqs):
        xv = widen(dyn.xv[s.vis_off:s.vis_off + s.n_frames * s.per_frame], "bf16")
        xa = widen(dyn.xa[s.aud_off:s.aud_off + s.n_audio], "bf16")
        xq = widen(dyn.xq[s.qry_off:s.qry_off + s.n_query], "bf16")
        r = OD.score_sequence(xv, xa, xq, s.n_frames, s.per_frame, dyn.params)
        m = r["margins"]
        assert min(m["gate"], m["segment"], m["segment_budget"], m["dafps"], m["dedup"]) > 1e-9, m
        assert m["frame_budget"] > (1e-4 if r["gate"] else 1e-9), m
        sl = slice(f0, f0 + s.n_frames)
        assert bool(got["gate"][i].item()) == r["gate"]
        np.testing.assert_array_equal(got["segment"][sl].cpu().numpy(), r["segment"])
        np.testing.assert_array_equal(got["budget"][sl].cpu().numpy(), r["frame_budget"])
        kept_all.append(r["kept"] + s.vis_off)
        f0 += s.n_frames
        log(f"  clip {i}: F={s.n_frames} gate={r['gate']} segments={r['g'].size} kept={r['kept'].size}")
    want = np.concatenate(kept_all)
    np.testing.assert_array_equal(got["kept"].cpu().numpy().astype(np.int64), want)
    return want


def _check_prune(prune, cache, out):
    sd = [dict(tok_off=s.tok_off, n_tokens=s.n_tokens, q_off=s.q_off, q_len=s.q_len, tags=s.tags(), keep=s.keep,
               keep_basis=s.keep_basis) for s in prune.seqs]
    w_scores, w_kept, w_n, margins = OP.prune_batch(widen(prune.q, "bf16"), widen(prune.k, "bf16"), sd)
    assert min(margins) >= 1e-2, margins
    assert out["n_kept"] == w_n
    np.testing.assert_array_equal(out["kept"].cpu().numpy().astype(np.int64), w_kept)
    g = out["scores"].cpu().numpy()
    for s in prune.seqs:
        sl = slice(s.tok_off, s.tok_off + s.n_tokens)
        c = s.tags() != 0
        rel = np.abs(g[sl][c] - w_scores[sl][c]) / w_scores[sl][c]
        assert rel.max() <= 2e-3
        assert np.all(g[sl][~c] == 0)
    kr = w_kept
    np.testing.assert_array_equal(bits(out["k_out"]), raw_bits(prune.k, "bf16")[:, kr])
    np.testing.assert_array_equal(bits(out["v_out"]), raw_bits(cache.v_layers[0], "bf16")[:, kr])
    np.testing.assert_array_equal(bits(out["h_out"]), raw_bits(cache.hidden, "bf16")[kr])
    np.testing.assert_array_equal(out["p_out"].cpu().numpy(), cache.pos[:, kr])


@pytest.mark.parametrize("structure", ["offset", "shared"])
def test_60s_clip_7b_shape_end_to_end(structure):
    log(f"[e2e] 60 s clip, 7B shape, {structure}")
    dyn = W.dynamics_cfg3(structure)
    prune = W.prune_cfg3()
    cache = W.cfg_cache(3, prune)
    out = _launch(dyn, prune, cache)
    kept_vis = _check_scorer(dyn, out["dyn"])
    np.testing.assert_array_equal(bits(out["emb"]), dyn.xv[kept_vis])
    _check_prune(prune, cache, out)


def test_ragged_batch_of_8_clips_end_to_end():
    log("[e2e] ragged batch of 8 clips, 20-300 s")
    rb = W.ragged_batch()
    log(f"  clip lengths (s): {rb.seconds}")
    out = _launch(rb.dynamics, rb.prune, rb.cache)
    kept_vis = _check_scorer(rb.dynamics, out["dyn"])
    np.testing.assert_array_equal(bits(out["emb"]), rb.dynamics.xv[kept_vis])
    _check_prune(rb.prune, rb.cache, out)
