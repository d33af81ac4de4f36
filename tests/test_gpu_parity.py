"""Parity of the HIP path (through the C ABI) with the fp64 oracle on small
workloads that still span several tiles, pages and ragged tails, plus the
paper's invariants evaluated on the GPU."""
import numpy as np
import pytest

from paper_2607_28940_amd import inputs as I
from paper_2607_28940_amd.inputs import ModelConfig
from tests.parity_util import BF16_TOL, FP32_TOL, DeviceCase, check_err, log, oracle_request, score_err, tensor_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    torch.cuda.set_device(0)


@pytest.fixture(scope="module")
def O(oracle_mod):
    return oracle_mod


def _compare_all(run: DeviceCase, orc, reqs, tol, label, append=False):
    g = run.score(reqs)
    o = [oracle_request(orc, run.wl, r, append=append)[0] for r in reqs]
    err = score_err(np.concatenate(g), np.concatenate(o))
    log(f"{label}: max err {err['max']:.3e} p99 {err['p99']:.3e} (tol {tol})")
    assert np.all(np.isfinite(np.concatenate(g)))
    check_err(err, tol)
    return g, o


@pytest.mark.parametrize("variant", [(), ("sharp", "affine")], ids=["base", "sharp-affine"])
def test_tiny_fp32(O, variant):
    wl = I.workload("tiny")
    w = I.make_weights(wl.model, variant)
    log(f"tiny fp32 {variant}")
    run = DeviceCase(wl, w)
    run.build([0])
    _compare_all(run, O.Oracle(wl.model, w), [0], FP32_TOL, f"tiny fp32 {variant}")


# bf16 models small enough for the oracle, shaped to hit the MFMA kernels
# (d_head 64 and 128), several 64-token pages with ragged last pages, query
# blocks with ragged tails, S = 0 and S > 64.
SMALL_BF16 = [
    ("dh128", ModelConfig(256, 2, 1024, 2, 2, rel_pos_buckets=16)),
    ("dh64", ModelConfig(256, 4, 512, 2, 2, rel_pos_buckets=16)),
    ("dh64-1dec-noRel", ModelConfig(512, 8, 1024, 1, 1, rel_pos_buckets=0)),
]
RAGGED = dict(L=[70, 200, 129, 1], S=[5, 0, 70, 3], C=[7, 100, 33, 1])


@pytest.mark.parametrize("name,model", SMALL_BF16, ids=[c[0] for c in SMALL_BF16])
def test_bf16_ragged_vs_oracle(O, name, model):
    wl = I.custom_workload(model, cfg_id=31, **RAGGED)
    w = I.make_weights(model, ("sharp", "affine"))
    log(f"bf16 ragged {name}")
    run = DeviceCase(wl, w)
    run.build(range(wl.B))
    _compare_all(run, O.Oracle(model, w), range(wl.B), BF16_TOL, f"bf16 ragged {name}")


def test_kv_split_vs_oracle(O):
    """Few requests with long caches: the cross-attention work list splits the
    long request's pages over several tiles per (head, query block) and merges
    their partial results (log-sum-exp), since a whole-request tile would leave
    the GPU idle (3000 cached tokens = 47 pages, in parts of at least 16). The
    scores match the oracle; reordering the candidates does not change the
    plan, and every candidate's scores are bitwise unchanged."""
    model = SMALL_BF16[0][1]
    wl = I.custom_workload(model, cfg_id=37, L=[3000, 40], S=[5, 3], C=[200, 10])
    w = I.make_weights(model, ("sharp", "affine"))
    run = DeviceCase(wl, w)
    run.build(range(wl.B))
    _compare_all(run, O.Oracle(model, w), range(wl.B), BF16_TOL, "kv-split")
    base = run.score([0, 1])
    cand = [I.request_tokens(wl, r, I.STREAM_CANDIDATES)[::-1].copy() for r in range(wl.B)]
    rev = run.score([0, 1], cand=cand)
    for r in range(wl.B):
        assert np.array_equal(rev[r], base[r][::-1]), r


# Enough rows for the persistent GEMM (M >= 2048 encoder and decoder rows,
# neither a multiple of its 256-row tile), at the smallest K it takes (256:
# the QKV, attention-output and FFN-up projections of a d = 256 model) and at
# K = 1024 (the FFN down-projection); 10 requests with ragged S, C and L.
GEMM_ROWS = dict(L=[211, 305, 177, 389, 260, 143, 330, 298, 155, 271], S=[3, 17, 40, 9, 0, 33, 12, 26, 5, 21],
                 C=[301, 188, 270, 155, 322, 240, 199, 167, 290, 216])


def test_persistent_gemm_ragged_rows(O):
    """The same calls run once in one pass (every large projection on the
    persistent kernel) and once with the smallest workspace (one request per
    pass, every projection on the per-tile kernel): both kernels sum each
    output in the same order, so the scores agree bitwise. Sampled requests
    are checked against the oracle (a tile or row mapped wrongly would move
    whole rows of scores by O(1))."""
    model = ModelConfig(256, 2, 1024, 2, 2, rel_pos_buckets=16)
    wl = I.custom_workload(model, cfg_id=61, **GEMM_ROWS)
    rows, enc_rows = sum(wl.S) + sum(wl.C), sum(wl.L)
    assert rows >= 2048 and rows % 256 and enc_rows >= 2048 and enc_rows % 256
    w = I.make_weights(model, ("sharp", "affine"))
    log(f"persistent GEMM rows: decoder {rows}, encoder {enc_rows}")
    big = DeviceCase(wl, w)
    big.build(range(wl.B))
    g = big.score(range(wl.B))
    small = DeviceCase(wl, w)
    small.build(range(wl.B), ws_limit=small.cache.workspace_min_bytes(0, wl.B, I.offsets(wl.L)))
    g1 = small.score(range(wl.B), ws_limit=small.cache.workspace_min_bytes(2, wl.B, I.offsets(wl.S),
                                                                            I.offsets(wl.C)))
    assert np.all(np.isfinite(np.concatenate(g)))
    assert np.array_equal(np.concatenate(g), np.concatenate(g1))
    reqs = [0, 3, 9]
    err = score_err(np.concatenate([g[r] for r in reqs]),
                    np.concatenate([oracle_request(O.Oracle(model, w), wl, r)[0] for r in reqs]))
    log(f"persistent GEMM ragged rows, requests {reqs}: max err {err['max']:.3e} p99 {err['p99']:.3e}")
    check_err(err, BF16_TOL)


def test_cache_contents_vs_oracle(O):
    model = SMALL_BF16[0][1]
    wl = I.custom_workload(model, cfg_id=32, L=[150, 64], S=[4, 4], C=[4, 4])
    w = I.make_weights(model, ("sharp", "affine"))
    run = DeviceCase(wl, w)
    run.build([0, 1])
    orc = O.Oracle(model, w)
    for r in (0, 1):
        _, st = oracle_request(orc, wl, r)
        for part, ref in ((0, st["K"]), (1, st["V"]), (2, st["Kx"]), (3, st["Vx"])):
            for layer in range(ref.shape[0]):
                g = run.cache.export(r, part, layer).float().cpu().numpy()
                e = tensor_err(g, ref[layer])
                log(f"cache r{r} part{part} layer{layer}: {e:.3e}")
                assert e < 2e-2, (r, part, layer, e)


@pytest.mark.parametrize("name,model", SMALL_BF16, ids=[m[0] for m in SMALL_BF16])
def test_append_equals_rebuild(O, name, model):
    """App. D remark: appending events through the incremental encoder gives the
    cache (and scores) of re-encoding the whole sequence. The appends (5, then
    8 events per request) run the encoder's causal attention on the
    register-streaming kernel (at most 32 new tokens per request), the rebuild
    on the LDS-staged one; head widths 128 and 64, with and without the
    relative-position bias."""
    wl = I.custom_workload(model, cfg_id=33, L=[60, 130], S=[6, 2], C=[9, 17], n_append=13)
    w = I.make_weights(model, ("sharp", "affine"))
    inc = DeviceCase(wl, w)
    inc.build([0, 1])
    inc.append([0, 1], 0, 5)     # 60 -> 65 crosses a page boundary
    inc.append([0, 1], 5, 13)
    assert inc.cache.length(0) == 73 and inc.cache.length(1) == 143
    full = DeviceCase(wl, w)
    X = [np.concatenate([I.request_tokens(wl, r, I.STREAM_BEHAVIOR), I.request_tokens(wl, r, I.STREAM_EVENTS)])
         for r in (0, 1)]
    full.cache.build([0, 1], full.dev(np.concatenate(X)), I.offsets([len(x) for x in X]))
    for r in (0, 1):
        for part in range(4):
            for layer in range(model.n_enc_layers if part < 2 else model.n_dec_layers):
                a = inc.cache.export(r, part, layer).float().cpu().numpy()
                b = full.cache.export(r, part, layer).float().cpu().numpy()
                e = tensor_err(a, b)
                log(f"append vs rebuild {name} r{r} part{part} layer{layer}: {e:.3e} exact={np.array_equal(a, b)}")
                assert e < 1e-2
    g_inc = np.concatenate(inc.score([0, 1]))
    g_full = np.concatenate(full.score([0, 1]))
    assert score_err(g_inc, g_full)["max"] < 1e-2
    orc = O.Oracle(model, w)
    o = np.concatenate([oracle_request(orc, wl, r, append=True)[0] for r in (0, 1)])
    err = score_err(g_inc, o)
    log(f"append scores vs oracle ({name}): {err}")
    check_err(err, BF16_TOL)


def test_candidates_independent_on_gpu():
    """Candidate scores do not depend on candidate order or on the other
    candidates sharing the request (bitwise on the GPU: every candidate row is
    computed by the same arithmetic wherever it sits)."""
    model = SMALL_BF16[1][1]
    wl = I.custom_workload(model, cfg_id=34, L=[100], S=[7], C=[150])
    w = I.make_weights(model, ("sharp",))
    run = DeviceCase(wl, w)
    run.build([0])
    Xc = I.request_tokens(wl, 0, I.STREAM_CANDIDATES)
    base = run.score([0], cand=[Xc])[0]
    perm = np.random.default_rng(1).permutation(len(Xc))
    assert np.array_equal(run.score([0], cand=[Xc[perm]])[0], base[perm])
    sub = np.array([3, 149, 77])
    assert np.array_equal(run.score([0], cand=[Xc[sub]])[0], base[sub])


def test_poisoned_pool_and_chunked_workspace():
    """Unused page slots full of NaN never reach the scores; running the call
    in several workspace-sized passes gives identical scores."""
    model = SMALL_BF16[0][1]
    wl = I.custom_workload(model, cfg_id=35, **RAGGED)
    w = I.make_weights(model, ("sharp",))
    clean = DeviceCase(wl, w, fill_byte=0)
    clean.build(range(wl.B))
    ref = np.concatenate(clean.score(range(wl.B)))
    dirty = DeviceCase(wl, w, fill_byte=0xFF, extra_pages=3)
    small = dirty.cache.workspace_min_bytes(0, wl.B, I.offsets(wl.L))
    dirty.build(range(wl.B), ws_limit=small)
    got = np.concatenate(dirty.score(range(wl.B)))
    assert np.all(np.isfinite(got))
    assert np.array_equal(got, ref)
    so, co = I.offsets(wl.S), I.offsets(wl.C)
    small = dirty.cache.workspace_min_bytes(2, wl.B, so, co)
    got2 = np.concatenate(dirty.score(range(wl.B), ws_limit=small))
    assert np.array_equal(got2, ref)


def test_status_codes_on_gpu():
    from paper_2607_28940_amd import transx as T
    model = SMALL_BF16[1][1]
    wl = I.custom_workload(model, cfg_id=36, L=[64, 65], S=[1, 1], C=[2, 2])
    w = I.make_weights(model)
    run = DeviceCase(wl, w, model_id=42, max_tokens=256)
    assert run.cache.model_id() == 42
    run.build([0, 1])
    assert run.cache.free_pages() == 0
    run.cache.release([1])
    assert run.cache.length(1) == -1 and run.cache.free_pages() == 2
    with pytest.raises(T.TxError) as ei:
        run.score([0, 1])
    assert ei.value.code == T.TX_E_NOCACHE
    with pytest.raises(T.TxError) as ei:
        run.append([0], 0, 1)  # wl.n_append == 0 -> empty event rows
    assert ei.value.code == T.TX_E_INVALID
    # pool exhausted: request 1 would need 2 pages plus 1 more for request 0
    X = np.concatenate([I.request_tokens(wl, 1, 0), I.request_tokens(wl, 1, 0)[:64]])
    with pytest.raises(T.TxError) as ei:
        run.cache.build([1], run.dev(X), I.offsets([len(X)]))
    assert ei.value.code == T.TX_E_NOMEM
    assert run.cache.length(1) == -1 and run.cache.free_pages() == 2
    # rebuild of a cached request replaces it in place
    run.build([0])
    assert run.cache.length(0) == 64 and run.cache.free_pages() == 2
    s = run.score([0])[0]
    assert np.all(np.isfinite(s))
