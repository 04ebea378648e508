"""Parity at the full widths of the benchmark shapes, one layer at a time.

Each case is a one-layer model made of a real layer of the seeded full-size
weights (same embedding, LM head and final gain), run through the C ABI over a
random committed bf16 cache installed with ``ee_load_kv``, and compared with
the oracle (Eq. 3's forward, Eq. 7's acceptance) on identical inputs:

* 7B (d 4096, 32 / 8 heads, FFN 11008, vocab 32256): layers 0, 15 and 31, a
  K = 32 block over 2048 committed positions; layer 15 with a 64-node draft
  tree (the tree walk and the compacted path checked too) and with
  entropy-aware top-5 verification (every clear threshold compared); layer
  31 with long drafts, K = 128 and 512;
* 1B (d 2048, 16 / 4 heads, FFN 5632): layer 7, a K = 16 block over 1024;
* 33B (d 7168, 56 / 8 heads: 7 query heads per KV head, FFN 19200): layer 30,
  one ``ee_verify_batch`` block of 4 sequences x 65 rows over 4096 committed
  positions each (260 rows: the split-K gate/up projection with a separate
  SwiGLU kernel, four K slices in the 7168-wide projections).

Every value the GPU rounds to bf16 (captured with ``ee_capture``: x_attn, q,
k, v, o, x_ffn, z, x_final) must be the oracle's rounding of the exact value,
or, where the exact value lies within a float32 evaluation's error of a bf16
rounding boundary, its other neighbour: both are correct results of the
definition, which the paper leaves to the evaluation's precision (reading
G20); the oracle then follows the GPU's choice.  With every rounding decision
checked, the logits of every row must match the oracle's within the stated
bf16 tolerance 2e-2, and in fact within 1e-4 (what is left is float32
accumulation in the unrounded paths: ~1.5e-6 measured), the committed K/V
must equal the oracle's bit for bit, and the accept length and next token
must be exactly the oracle's wherever the margins decide them.  The flips
are rare (~4e-4 of the values; at most 2e-3 allowed, which a biased kernel
would exceed).

Without following the near-tie choices, the oracle's own rounding differs
from the GPU's at those few hundred values per block, and each flip moves
later rounded values across their boundaries, so the logits differ by
0.014-0.028 at one layer (and ~0.12 through 32 layers, test_gpu_fullsize.py):
printed, and held only to a loose 0.1 here, since it measures the model's
sensitivity to rounding flips rather than the kernels.
"""

import numpy as np
import pytest

from helpers import OneLayer, RoundingCheck, deciding_margin, gpu_site_values
from oracle import OracleSession, greedy_rows, top2_margin
from oracle.numerics import to_f64
from workloads import gen_weights, get_shape, random_kv_context, random_tree, zipf_tokens

pytestmark = pytest.mark.gpu

TOL = 2e-2          # the stated bf16 logit tolerance
TIGHT = 1e-4        # logits once the rounding decisions are checked and followed
LOOSE = 0.1         # logits of the oracle's own rounding (the flip cascade)


@pytest.fixture(scope="module")
def ee():
    import paper_2506_02780_amd as mod
    return mod


def _case(name, layer):
    full = get_shape(name)
    w = gen_weights(full, seed=1234, eager=False)
    return full.with_(n_layers=1), OneLayer(w, layer)


def _install(eng, shape, b, ctx, seed):
    kv = random_kv_context(1, ctx, shape.n_kv_heads, shape.head_dim, seed=seed, dtype="bf16")
    pending = int(zipf_tokens(shape.vocab, 1, seed=seed + 100)[0])
    eng.load_kv(b, np.stack([k for k, _ in kv]), np.stack([v for _, v in kv]), pending)
    return [(to_f64(k, "bf16"), to_f64(v, "bf16")) for k, v in kv], pending


def _compare(shape, w, cache, pending, draft, gpu_logits, gpu_a, gpu_next, sites, gpu_kv, label, parent=None):
    """Oracle twice: checking and following the GPU's rounding decisions
    (logits within 2e-2 and 1e-4, K/V bitwise), and with its own rounding
    (the flip cascade: printed, held to 0.1).  parent: a draft tree."""
    ref = OracleSession(shape, w)
    ref.set_cache(cache, pending)
    ra, rn, _ = ref.verify(draft, parent)
    plain = float(np.abs(gpu_logits - ref.last_logits).max())
    chk = RoundingCheck(sites)
    fol = OracleSession(shape, w, rounding=chk)
    fol.set_cache(cache, pending)
    fa, fn, fpath = fol.verify(draft, parent)
    tight = float(np.abs(gpu_logits - fol.last_logits).max())
    print(f"[fullwidth] {label}: |GPU - oracle| {plain:.4f}, after checked rounding {tight:.2e}; "
          f"{chk.summary()}; accept {gpu_a}/{ra}, next {gpu_next}/{rn}", flush=True)
    assert chk.mismatches() == 0, chk.summary()
    assert chk.flips() <= 2e-3 * chk.values(), chk.summary()
    assert tight <= TOL and tight <= TIGHT
    assert plain <= LOOSE
    # acceptance, decided on the checked logits: exact wherever the deciding
    # rows' top-2 margins exceed the remaining difference (a tree walk is
    # decided by the rows it visits: the pending row and the accepted path)
    decide = (deciding_margin(fol.last_logits, fa, len(draft)) if parent is None
              else float(top2_margin(fol.last_logits[[0] + list(fpath)]).min()))
    if decide > TIGHT:
        assert (gpu_a, gpu_next) == (fa, fn)
    # committed K/V: the pending row and the accepted rows, bit for bit
    n = cache[0][0].shape[0]
    gk, gv = gpu_kv
    fk = fol.cache[0][0][n:]
    fv = fol.cache[0][1][n:]
    assert gk.shape == fk.shape == (1 + gpu_a, shape.n_kv_heads, shape.head_dim)
    assert np.array_equal(gk, fk) and np.array_equal(gv, fv)
    return fol


def _single(ee, name, layer, ctx, k, seed):
    shape, w = _case(name, layer)
    eng = ee.Engine(shape, w, max_ctx=ctx + k + 8, k_max=k)
    try:
        cache, pending = _install(eng, shape, 0, ctx, seed)
        draft = zipf_tokens(shape.vocab, k, seed=seed + 1)
        for blk in range(2):
            eng.rollback(0, ctx, pending)
            eng.capture(k + 1)
            a, nxt, _ = eng.verify(0, draft)
            eng.capture(None)
            lg = eng.logits()
            sites = gpu_site_values(eng.captured(), shape, slice(0, k + 1))
            kk, vv = eng.read_kv(0, 0)
            gkv = (to_f64(kk[ctx:], "bf16"), to_f64(vv[ctx:], "bf16"))
            fol = _compare(shape, w, cache, pending, draft, lg, a, nxt, sites, gkv,
                           f"{name} layer {layer} K={k} n={ctx} block {blk}")
            # second block: the first draft token replaced by the greedy one,
            # so at least one draft token is accepted
            draft = np.concatenate([[greedy_rows(fol.last_logits)[0]], draft[1:]]).astype(np.int32)
        assert a >= 1
    finally:
        eng.close()


@pytest.mark.parametrize("layer", [0, 15, 31])
def test_7b_layer_k32_over_2048_positions(ee, layer):
    _single(ee, "7b", layer, 2048, 32, seed=50 + layer)


def test_1b_layer_k16_over_1024_positions(ee):
    _single(ee, "1b", 7, 1024, 16, seed=70)


def test_7b_layer_entropy_topk_over_2048_positions(ee):
    """Entropy-aware verification (Eq. 9-10, k = 5) at the 7B width: the
    block's rounding decisions checked and followed as above, then every
    threshold tau compared with the oracle's wherever the top-6 logit gaps and
    k H's distance to an integer exceed the remaining difference, and the
    outcome where every deciding row is clear.  Second block: the first
    three draft tokens replaced by their row's second-best token, which
    Eq. 10 accepts whenever tau >= 2."""
    from oracle import entropy_threshold
    shape, w = _case("7b", 15)
    ctx, k, top = 2048, 32, 5
    eng = ee.Engine(shape, w, max_ctx=ctx + k + 8, k_max=k)
    try:
        cache, pending = _install(eng, shape, 0, ctx, seed=85)
        draft = zipf_tokens(shape.vocab, k, seed=86)
        compared = 0
        for blk in range(2):
            eng.rollback(0, ctx, pending)
            eng.capture(k + 1)
            (a, nxt, thr), = eng.verify_topk([0], [draft], top, True)
            eng.capture(None)
            lg = eng.logits()
            chk = RoundingCheck(gpu_site_values(eng.captured(), shape, slice(0, k + 1)))
            fol = OracleSession(shape, w, rounding=chk)
            fol.set_cache(cache, pending)
            fa, fn, _ = fol.verify_topk(draft, top, True)
            tight = float(np.abs(lg - fol.last_logits).max())
            print(f"[fullwidth] 7b layer 15 top-{top} K={k} block {blk}: after checked rounding {tight:.2e}; "
                  f"{chk.summary()}; accept {a}/{fa}, next {nxt}/{fn}", flush=True)
            assert chk.mismatches() == 0, chk.summary()
            assert tight <= TIGHT
            clear = []
            for i in range(k + 1):
                s = np.sort(fol.last_logits[i])[::-1][:top + 1]
                _, h, tau = entropy_threshold(fol.last_logits[i], top)
                x = top * h
                ok = np.min(s[:-1] - s[1:]) > 2 * tight and abs(x - round(x)) > 15 * tight
                clear.append(ok)
                if ok and i < k:
                    assert thr[i] == tau, (blk, i, thr[i], tau)
                    compared += 1
            if all(clear[:fa + 1]):
                assert (a, nxt) == (fa, fn)
            second = np.argsort(-fol.last_logits, axis=1, kind="stable")[:, 1]
            draft = draft.copy()
            draft[:3] = second[:3]
        assert a >= 1 and compared >= 32
    finally:
        eng.close()


@pytest.mark.parametrize("k", [128, 512])
def test_7b_layer_long_draft_over_2048_positions(ee, k):
    """Long Reuse drafts at the 7B width: the fused projections in 32-row
    groups (5 and 16 of them), the down projection and LM head in 80-row
    groups, the wide attention kernel (33 and 129 query tiles)."""
    _single(ee, "7b", 31, 2048, k, seed=60 + k)


def test_7b_layer_tree64_over_2048_positions(ee):
    """A 64-node draft tree (depth 8, branching 3) at the 7B width over 2048
    positions: 17 query tiles, so the tree's split and the splits below it run
    in one launch.  Second block: the root's first child replaced by the
    greedy token, so the walk accepts at least one node."""
    shape, w = _case("7b", 15)
    ctx, k = 2048, 64
    eng = ee.Engine(shape, w, max_ctx=ctx + k + 8, k_max=k)
    try:
        cache, pending = _install(eng, shape, 0, ctx, seed=80)
        parent = random_tree(k, max_depth=8, max_branch=3, seed=11)
        draft = zipf_tokens(shape.vocab, k, seed=81)
        first = int(np.flatnonzero(parent == -1)[0])   # the root's first child
        for blk in range(2):
            eng.rollback(0, ctx, pending)
            eng.capture(k + 1)
            a, nxt, _ = eng.verify(0, draft, parent)
            eng.capture(None)
            lg = eng.logits()
            sites = gpu_site_values(eng.captured(), shape, slice(0, k + 1))
            kk, vv = eng.read_kv(0, 0)
            gkv = (to_f64(kk[ctx:], "bf16"), to_f64(vv[ctx:], "bf16"))
            fol = _compare(shape, w, cache, pending, draft, lg, a, nxt, sites, gkv,
                           f"7b layer 15 tree of {k} nodes n={ctx} block {blk}", parent=parent)
            draft = draft.copy()
            draft[first] = greedy_rows(fol.last_logits)[0]
        assert a >= 1
    finally:
        eng.close()


def test_33b_layer_batch_of_4_k64_over_4096_positions(ee):
    """Four sequences in one ee_verify_batch block of 260 rows; each sequence
    is checked against its own oracle session."""
    shape, w = _case("33b", 30)
    B, K, CTX = 4, 64, 4096
    eng = ee.Engine(shape, w, max_ctx=CTX + K + 8, max_seqs=B, k_max=K)
    try:
        caches, pendings, drafts = [], [], []
        for b in range(B):
            c, p = _install(eng, shape, b, CTX, seed=90 + b)
            caches.append(c)
            pendings.append(p)
            drafts.append(zipf_tokens(shape.vocab, K, seed=95 + b))
        eng.capture(B * (K + 1))
        res = eng.verify_batch(list(range(B)), drafts)
        eng.capture(None)
        lg = eng.logits()
        cap = eng.captured()
        for b in range(B):
            rows = slice(b * (K + 1), (b + 1) * (K + 1))
            a, nxt, _ = res[b]
            kk, vv = eng.read_kv(b, 0)
            gkv = (to_f64(kk[CTX:], "bf16"), to_f64(vv[CTX:], "bf16"))
            _compare(shape, w, caches[b], pendings[b], drafts[b], lg[rows], a, nxt,
                     gpu_site_values(cap, shape, rows), gkv, f"33b layer 30 batch seq {b}")
    finally:
        eng.close()
