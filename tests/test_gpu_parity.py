"""GPU parity: the HIP library against the CPU oracle on the five workloads.

Selections, masks, the retrospective mask A and sequence lengths must match
bit for bit every step; outputs and log-normalisers within 2e-3 max-abs for
bf16 inputs (fp32 accumulation) and 1e-5 for fp32 inputs.  Steps are fewer
than the full workloads where the oracle would take minutes; each run still
spans many tiles, splits and a ragged last page, and covers the window's
ramp-up and several wraps of the output-cache ring.
"""
import pytest

import workloads as W
from gpu_harness import run_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_09001_amd import binding
    binding.load_library()


def test_tiny_fp32_all_steps():
    run_parity(W.config(0), W.config(0).steps)


def test_tiny_fp32_separate_entry_points():
    run_parity(W.config(0), 12, split_calls=True, label="tiny-fp32 split calls")


def test_tiny_fp32_shuffled_page_table():
    run_parity(W.config(0), 12, page_perm_seed=5, label="tiny-fp32 shuffled pages")


def test_llama_layer_32k():
    spec = W.config(1)
    run_parity(spec, 40)


def test_llama_layer_32k_split_calls_shuffled():
    spec = W.config(1)
    run_parity(spec, 20, split_calls=True, page_perm_seed=1, label="32k split+shuffled")


@pytest.mark.timeout(900)
def test_batched_serving_ragged():
    """All 128 steps of the batch-16 workload (ragged 8K-32K contexts, shuffled
    page table): selection, mask, last_loaded, seq_lens and page scores bit for
    bit, every output row against the oracle's."""
    spec = W.config(2)
    run_parity(spec, spec.steps, page_perm_seed=2, label="batch16 ragged shuffled, all steps")


@pytest.mark.timeout(900)
def test_long_generation_multi_token_steps():
    """The long-generation workload at its full batch of 4, 8 tokens appended per
    step (16384 -> 16896 tokens over these 64 steps), every output row against the
    oracle's."""
    spec = W.config(3)
    run_parity(spec, 64, label="long-generation b4 8 tok/step, 64 steps")


@pytest.mark.parametrize("budget,window", [(1024, 0), (2048, 4), (4096, 16), (8192, 64)])
def test_extreme_context_sweep(budget, window):
    spec = W.config(4).replace(budget=budget, window=window)
    run_parity(spec, 10, label=f"131k B={budget} W={window}")


@pytest.mark.parametrize("window", [0, 4])
def test_extreme_context_full_budget_is_dense(window):
    # budget covering the whole context: every page selected, current row = dense
    spec = W.config(4).replace(budget=131072 + 4096, window=window)
    run_parity(spec, 3, label=f"131k dense W={window}")


def test_short_sequences_and_partial_pages():
    # sequences shorter than one page and budgets above the context
    spec = W.Spec("edge-short", batch=3, num_kv_heads=2, group=3, head_dim=64, page_size=16,
                  budget=64, window=5, steps=20, dtype="bf16", prefill=(1, 17, 40), seed=9)
    run_parity(spec, 20, page_perm_seed=3, label="edge short")


def test_group_one_wide_window():
    spec = W.Spec("edge-w64-g1", batch=2, num_kv_heads=1, group=1, head_dim=128, page_size=32,
                  budget=256, window=64, steps=70, dtype="bf16", prefill=(500, 900), seed=10)
    run_parity(spec, 70, label="edge W=64 G=1")


def test_fp32_head_dim_128_many_rows():
    spec = W.Spec("edge-f32-d128", batch=1, num_kv_heads=2, group=8, head_dim=128, page_size=16,
                  budget=512, window=20, steps=24, dtype="f32", prefill=(3000,), seed=12)
    run_parity(spec, 24, label="edge f32 d128 R=168")


def test_six_row_tiles_bf16_d64():
    # R = 23 * 4 = 92 rows: six 16-row tiles, more than the four SIMDs of a CU
    spec = W.Spec("edge-6tiles", batch=2, num_kv_heads=2, group=4, head_dim=64, page_size=16,
                  budget=640, window=22, steps=28, dtype="bf16", prefill=(2100, 1337), seed=13)
    run_parity(spec, 28, page_perm_seed=4, label="edge 6 row tiles bf16 d64")


def test_five_row_tiles_fp32():
    # R = 35 * 2 = 70 rows: five tiles, fp32 inputs
    spec = W.Spec("edge-5tiles-f32", batch=1, num_kv_heads=2, group=2, head_dim=128, page_size=16,
                  budget=384, window=34, steps=40, dtype="f32", prefill=(1500,), seed=14)
    run_parity(spec, 40, label="edge 5 row tiles f32")


def test_step_attend_partials_entry_point():
    """The timing entry point of the step's scores + selection + attention
    launch, run after a step (same query row, the token now stored), selects
    the same pages; its mask values are last_loaded as the step left it, which
    it does not change."""
    import numpy as np
    import torch
    from gpu_harness import _gpu_layer
    spec = W.config(1)
    gen = W.Generator(spec)
    layer = _gpu_layer(spec, 6)
    for b, (k, v) in enumerate(gen.prefill()):
        layer.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    for t in range(6):
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        for j in range(k_new.shape[0] - 1):
            layer.append(t, k_new[j], v_new[j])
        layer.step(t, win, k_new[-1], v_new[-1])
    torch.cuda.synchronize()
    sel0 = layer.selected.cpu().numpy().copy()
    num0 = layer.num_selected.cpu().numpy().copy()
    A0 = layer.last_loaded.cpu().numpy().copy()
    print(f"[entry] retro_step_attend_partials after step {t}", flush=True)
    layer.step_attend_partials(t, layer._dev(win))
    torch.cuda.synchronize()
    assert np.array_equal(layer.num_selected.cpu().numpy(), num0)
    assert np.array_equal(layer.selected.cpu().numpy(), sel0)
    assert np.array_equal(layer.last_loaded.cpu().numpy(), A0)
    msk = layer.mask.cpu().numpy()
    want = np.full_like(sel0, -1)
    for b in range(sel0.shape[0]):
        for h in range(sel0.shape[1]):
            k = int(num0[b, h])
            want[b, h, :k] = A0[b, h, sel0[b, h, :k]]
    assert np.array_equal(msk, want)


def test_attention_wait_timeout_leaves_state_untouched():
    """Failure path of the two-launch step, forced from the host through
    RETRO_FLAG_TEST_WAIT_TIMEOUT: every wait between the workgroups of the first
    launch gives up after a few polls (its awaited tag out of reach), so every
    workgroup still runs to its end.  The step's outputs must be NaN, and the
    output cache, last_loaded and seq_lens exactly as before the step; the error
    word is sticky, so the next call fails the same way with normal waits; once
    the workspace is zero-filled the step is retried and matches the oracle."""
    import numpy as np
    import oracle
    import torch
    from gpu_harness import TOL, Stats, _gpu_layer, compare_step
    from paper_2508_09001_amd import binding as B
    spec = W.config(0)
    gen = W.Generator(spec)
    orc = oracle.Oracle.for_spec(spec)
    layer = _gpu_layer(spec, None)
    for b, (k, v) in enumerate(gen.prefill()):
        orc.prefill(b, k, v)
        layer.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    stats = Stats()
    for t in range(spec.window + 3):
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        ref = orc.step(t, k_new, v_new, win)
        ref["A"] = orc.A
        if t == spec.window + 2:  # the ring is full: every slot has state to corrupt
            before = {n: getattr(layer, n).clone() for n in
                      ("o_cache", "lse_cache", "last_loaded", "seq_lens")}
            for forced in (True, False):
                layer.dims.flags = B.RETRO_FLAG_TEST_WAIT_TIMEOUT if forced else 0
                print(f"[timeout] step {t} forced={forced}", flush=True)
                layer.step(t, win, k_new[-1], v_new[-1])
                layer.dims.flags = 0
                torch.cuda.synchronize()
                assert torch.isnan(layer.o_out).all() and torch.isnan(layer.lse_out).all()
                for n, v in before.items():
                    assert torch.equal(getattr(layer, n), v), f"{n} changed by a failed step"
                layer._lens = [int(x) for x in before["seq_lens"].cpu()]
            layer.workspace.zero_()
        print(f"[timeout] step {t}", flush=True)
        layer.step(t, win, k_new[-1], v_new[-1])
        compare_step(t, layer, ref, TOL[spec.dtype], stats)


def test_workspace_of_another_geometry_is_refused():
    """A workspace last used by the one-launch step of another geometry (here the
    headline layer with W = 16, then W = 4) is refused: outputs NaN, the second
    layer's output cache, last_loaded and seq_lens untouched."""
    import numpy as np
    import torch
    from gpu_harness import _gpu_layer
    spec_a = W.config(1)
    spec_b = W.config(1).replace(window=4)
    la, lb = _gpu_layer(spec_a, None), _gpu_layer(spec_b, None)
    assert lb.ws_bytes <= la.ws_bytes
    gen_a, gen_b = W.Generator(spec_a), W.Generator(spec_b)
    for b, (k, v) in enumerate(gen_a.prefill()):
        la.prefill(b, k, v)
    for b, (k, v) in enumerate(gen_b.prefill()):
        lb.prefill(b, k, v)
    qa, qb = W.QueryWindow(spec_a), W.QueryWindow(spec_b)
    for t in range(2):
        k_new, v_new, q = gen_a.step(t)
        la.step(t, qa.push(q).copy(), k_new[-1], v_new[-1])
    torch.cuda.synchronize()
    assert torch.isfinite(la.o_out).all()
    lb.workspace = la.workspace  # the same scratch, now for another geometry
    before = {n: getattr(lb, n).clone() for n in ("o_cache", "lse_cache", "last_loaded",
                                                  "seq_lens")}
    k_new, v_new, q = gen_b.step(0)
    print("[geometry] step 0 of W = 4 on a W = 16 workspace", flush=True)
    lb.step(0, qb.push(q).copy(), k_new[-1], v_new[-1])
    torch.cuda.synchronize()
    # the one-launch step's per-workgroup control lines (launch count,
    # fingerprint, failure mark), for the failure messages: a workgroup that
    # refused the workspace counts 3 launches, one that took it as fresh 1
    lines = lb.workspace[:1024 * 128].view(torch.int32).view(1024, 32)[:, :4].cpu().numpy()
    info = (f"launch counts {np.unique(lines[:, 0], return_counts=True)}, fingerprints "
            f"{np.unique(lines[:, 2], return_counts=True)}, marks {np.unique(lines[:, 3])}")
    assert torch.isnan(lb.o_out).all() and torch.isnan(lb.lse_out).all(), info
    for n, v in before.items():
        now = getattr(lb, n)
        diff = torch.nonzero(now != v)
        assert diff.numel() == 0, (f"{n} changed by a refused step at {diff.shape[0]} entries "
                                   f"(NaN before the step: {bool(torch.isnan(v).any()) if v.is_floating_point() else False}), "
                                   f"first {diff[:4].tolist()}: {now[tuple(diff[:4].T)].tolist()} "
                                   f"(was {v[tuple(diff[:4].T)].tolist()}); {info}")


def test_launch_epoch_wraps():
    """The one-launch step's epochs run 1 .. 2^31 - 1 and then start again at 1.
    A fresh workspace whose control lines (set from the host) say that the last
    launch had epoch 2^31 - 2: the next steps run at epochs 2^31 - 1, 1, 2, ...
    and must match the oracle bit for bit (selections) and within tolerance
    (outputs) across the wrap."""
    import numpy as np
    import oracle
    import torch
    from gpu_harness import TOL, Stats, _gpu_layer, compare_step
    from paper_2508_09001_amd import binding as B
    for cfg in (0, 1):
        spec = W.config(cfg)
        gen = W.Generator(spec)
        orc = oracle.Oracle.for_spec(spec)
        layer = _gpu_layer(spec, None)
        assert B.retro_step_launches(layer.dims) == 1
        for b, (k, v) in enumerate(gen.prefill()):
            orc.prefill(b, k, v)
            layer.prefill(b, k, v)
        lines = layer.workspace[:1024 * 128].view(torch.int32).view(1024, 32)
        lines[:, 0] = 0x7FFFFFFE
        lines[:, 1] = 0
        qw = W.QueryWindow(spec)
        stats = Stats()
        for t in range(spec.window + 3):
            k_new, v_new, q = gen.step(t)
            win = qw.push(q).copy()
            ref = orc.step(t, k_new, v_new, win)
            ref["A"] = orc.A
            print(f"[epoch wrap] {spec.name} step {t}", flush=True)
            layer.step(t, win, k_new[-1], v_new[-1])
            compare_step(t, layer, ref, TOL[spec.dtype], stats)
            # the lines of the launch's workgroups hold its epoch; the rest
            # (no workgroup of this geometry) keep the preset value
            epochs = set(np.unique(lines[:, 0].cpu().numpy()).tolist())
            want = 0x7FFFFFFF if t == 0 else t
            assert int(lines[0, 0]) == want and epochs <= {want, 0x7FFFFFFE}, (t, epochs)


def test_token_page_on_physical_page_zero_with_a_grid_off_the_xcd_count():
    """Three KV heads of three splits each (9 workgroups: not a multiple of the 8
    XCDs, so workgroups keep their dispatch order), the step's token pages mapped
    to physical page 0 and its neighbour, the rest shuffled: the token's key and
    value reach the gather of their own step from the step's input, whatever the
    cache line of physical page 0 holds."""
    import numpy as np
    from paper_2508_09001_amd import binding as B
    from gpu_harness import _gpu_layer
    spec = W.Spec(name="grid9", batch=1, num_kv_heads=3, group=2, head_dim=64, page_size=16,
                  budget=80, window=3, steps=24, dtype="bf16", prefill=(400,), seed=41)
    mp = spec.max_pages
    rng = np.random.default_rng(5)
    pt = rng.permutation(mp).astype(np.int32)
    first = spec.prefill[0] // spec.page_size  # the page the first steps append to
    for lp, ph in ((first, 0), (first + 1, 1)):
        j = int(np.where(pt == ph)[0][0])
        pt[j], pt[lp] = pt[lp], pt[j]
    layer = _gpu_layer(spec, None, page_table=pt[None])
    assert B.retro_step_launches(layer.dims) == 1
    del layer
    run_parity(spec, spec.steps, page_table=pt[None], label="9 workgroups, token on page 0")


@pytest.mark.parametrize("budget,prefill,hk", [(512, 32000, 8), (512, 40000, 2)])
def test_long_context_shape_of_the_one_launch_step(budget, prefill, hk):
    """The one-launch step's long-context shape (ten selection stripes per
    thread, five score passes) away from the 131K workload: a small budget that
    leaves few splits, so that each workgroup scores more than 96 pages of a
    2000-page sequence, and a 2500-page sequence on two KV heads."""
    from paper_2508_09001_amd import binding as B
    from gpu_harness import _gpu_layer
    spec = W.Spec(name=f"long-shape-{budget}", batch=1, num_kv_heads=hk, group=4, head_dim=128,
                  page_size=16, budget=budget, window=8, steps=10, dtype="bf16",
                  prefill=(prefill,), seed=budget + hk)
    layer = _gpu_layer(spec, None)
    assert B.retro_step_launches(layer.dims) == 1
    del layer
    run_parity(spec, spec.steps, page_perm_seed=7, label=f"long shape B={budget} hk={hk}")


def test_page_pool_larger_than_the_tables_shuffled():
    """Physical pages drawn at random from a pool larger than batch * max_pages
    (digests stay per logical page): the headline layer and a ragged batch."""
    spec = W.config(1)
    run_parity(spec, 12, page_perm_seed=11, pool_pages=spec.batch * spec.max_pages + 3001,
               label="32k, pool +3001 pages, shuffled")
    spec = W.config(2)
    run_parity(spec, 6, page_perm_seed=12, pool_pages=spec.batch * spec.max_pages + 517,
               label="batch16, pool +517 pages, shuffled")


def test_relative_budget_grows_with_context():
    # relative budget of 0.15 with a 256-token floor: sequence 1 crosses from
    # 16 to 17 pages per step (0.15 * 1814 = 272.1 tokens) during the run
    spec = W.Spec("relative-budget", batch=2, num_kv_heads=2, group=4, head_dim=128, page_size=16,
                  budget=256, window=4, steps=20, dtype="bf16", prefill=(1700, 1810), seed=21,
                  budget_permille=150)
    run_parity(spec, 20, page_perm_seed=7, label="relative budget 0.15, min 256")


def test_relative_budget_llama_layer_32k():
    # the headline layer with the paper's relative budget: 307+ pages per step
    spec = W.config(1).replace(budget_permille=150)
    run_parity(spec, 10, label="32k relative budget 0.15")


def test_update_kv_tiny_fp32():
    # UpdateKV of the W = 4 past tokens before every step (Alg. 1 order)
    run_parity(W.config(0), 16, update_kv=True, label="tiny-fp32 + UpdateKV")


def test_update_kv_llama_layer_32k():
    run_parity(W.config(1), 10, page_perm_seed=3, update_kv=True, label="32k + UpdateKV")


def test_update_kv_short_sequences_and_partial_pages():
    spec = W.Spec("edge-short", batch=3, num_kv_heads=2, group=3, head_dim=64, page_size=16,
                  budget=64, window=5, steps=20, dtype="bf16", prefill=(1, 17, 40), seed=9)
    run_parity(spec, 20, page_perm_seed=3, update_kv=True, label="edge short + UpdateKV")


@pytest.mark.parametrize("f", [2, 3])
def test_topk_reuse_tiny_fp32(f):
    """The selection-reuse baseline (top-k refreshed every f steps): selection,
    mask, last_loaded and seq_lens bit for bit, outputs within tolerance, on every
    step of the tiny workload, through retro_step and through the separate calls."""
    spec = W.config(0).replace(reuse_interval=f)
    run_parity(spec, spec.steps, label=f"tiny fp32, top-k reuse f={f}")
    run_parity(spec, 12, split_calls=True, page_perm_seed=3,
               label=f"tiny fp32, top-k reuse f={f}, separate calls")


def test_topk_reuse_llama_layer_32k():
    """Top-k reuse with f = 2 at the 32K layer: refresh steps take the one-launch
    step, reuse steps the append + mask + attention + merge launches."""
    spec = W.config(1).replace(reuse_interval=2)
    run_parity(spec, spec.window + 9, page_perm_seed=8, label="32k, top-k reuse f=2")

