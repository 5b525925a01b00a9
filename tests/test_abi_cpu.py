"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, its pure helpers return the documented values, and invalid
arguments are rejected on the host before anything is launched."""
import ctypes
import os
import re

import pytest

from paper_2606_09508_amd import binding as eb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "entropyinfer.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ei_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(eb.LIB_PATH):
        pytest.skip("libentropyinfer.so is not built")
    return eb.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert {"ei_entropy_probe", "ei_select_blocks", "ei_sparse_prefill_attn",
            "ei_dense_prefill_attn"} <= set(names)
    for n in names:
        assert hasattr(L, n), f"{n} declared in the header but not exported"


def test_helpers(L):
    assert L.ei_abi_version() == 7
    assert eb.kmax(128, 64, 2048, 3) == 98
    assert eb.kmax(2048, 64, 2048, 3) == 96 + 32
    assert eb.kmax(256, 128, 256, 3) == 6 + 2
    d = eb.Dims(1, 32, 8, 131072, 128)
    assert L.ei_num_segments(d, eb.Tiling(128, 64)) == 1024
    assert L.ei_num_blocks(d, eb.Tiling(128, 64)) == 2048
    assert L.ei_num_segments(eb.Dims(1, 4, 1, 1000, 128), eb.Tiling(128, 64)) == 8
    assert L.ei_num_blocks(eb.Dims(1, 4, 1, 1000, 128), eb.Tiling(128, 64)) == 16
    ws = L.ei_probe_workspace_bytes(d, eb.Tiling(128, 64))
    assert ws >= 32 * 1024 * 2 * 128 * 8 + 8 * 2048 * 2 * 128 * 2
    assert L.ei_probe_workspace_bytes(eb.Dims(1, 4, 1, 1024, 64), eb.Tiling(128, 64)) == 0
    for st in (0, -1, -2, -3, -4, -5):
        assert L.ei_status_str(st).decode().startswith(eb._STATUS[st])


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation


@pytest.mark.parametrize("dims,tiling,expect", [
    (eb.Dims(1, 4, 1, 1024, 64), eb.Tiling(128, 64), -3),     # D != 128
    (eb.Dims(1, 6, 4, 1024, 128), eb.Tiling(128, 64), -2),    # Hq % Hkv
    (eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 32), -3),    # L_B not 64/128
    (eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(192, 64), -2),    # L_S not a multiple of 128
    (eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 256), -3),   # L_B not 64/128
    (eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(64, 64), -2),     # L_S below 128
    (eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(0, 64), -2),
    (eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(-128, 64), -2),
    (eb.Dims(-1, 4, 1, 1024, 128), eb.Tiling(128, 64), -2),
    (eb.Dims(1, 0, 1, 1024, 128), eb.Tiling(128, 64), -2),
])
def test_probe_rejects_bad_shapes(L, dims, tiling, expect):
    st = L.ei_entropy_probe(FAKE, FAKE, dims, tiling, 1.0, FAKE, FAKE, FAKE, 1 << 30, None)
    assert st == expect


def test_probe_null_and_workspace(L):
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    assert L.ei_entropy_probe(None, FAKE, d, t, 1.0, FAKE, FAKE, FAKE, 1 << 30, None) == -1
    assert L.ei_entropy_probe(FAKE, FAKE, d, t, 1.0, None, FAKE, FAKE, 1 << 30, None) == -1
    need = L.ei_probe_workspace_bytes(d, t)
    assert L.ei_entropy_probe(FAKE, FAKE, d, t, 1.0, FAKE, FAKE, FAKE, need - 1, None) == -4
    assert L.ei_entropy_probe(FAKE, FAKE, d, t, 1.0, FAKE, FAKE, None, need, None) == -4
    assert L.ei_entropy_probe(FAKE, FAKE, d, t, float("nan"), FAKE, FAKE, FAKE, need, None) == -2


def test_empty_problems_launch_nothing(L):
    t = eb.Tiling(128, 64)
    for d in (eb.Dims(0, 4, 1, 1024, 128), eb.Dims(1, 4, 1, 0, 128)):
        assert L.ei_entropy_probe(None, None, d, t, 1.0, None, None, None, 0, None) == 0
        assert L.ei_select_blocks(None, None, d, t, eb.budget_params(), 98, None, None, None,
                                  None, None) == 0
        assert L.ei_sparse_prefill_attn(None, None, None, d, t, 0.088, None, None, 98, None,
                                        None, 0, None) == 0
        assert L.ei_dense_prefill_attn(None, None, None, d, 0.088, 1, None, None) == 0


def test_select_rejects_bad_params(L):
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    p = eb.budget_params(base_budget=256)
    km = L.ei_kmax(t, p)
    args = (FAKE,) * 5
    assert L.ei_select_blocks(FAKE, FAKE, d, t, p, km - 1, *args) == -2
    assert L.ei_select_blocks(FAKE, FAKE, d, t, eb.budget_params(base_budget=-1), km, *args) == -2
    assert L.ei_select_blocks(FAKE, FAKE, d, t, eb.budget_params(mult=0), km, *args) == -2
    assert L.ei_select_blocks(FAKE, FAKE, d, t, eb.budget_params(alpha=float("nan")), km,
                              *args) == -2
    assert L.ei_select_blocks(FAKE, None, d, t, p, km, *args) == -1
    assert L.ei_select_blocks(FAKE, FAKE, d, t, p, km, FAKE, FAKE, None, FAKE, None) == -1
    for mode in (-1, 3, 100):
        assert L.ei_select_blocks_mode(FAKE, FAKE, d, t, p, mode, km, *args) == -2
    assert L.ei_select_blocks_mode(FAKE, FAKE, d, t, p, 1, km - 1, *args) == -2
    assert L.ei_select_blocks_mode(FAKE, None, d, t, p, 2, km, *args) == -1


def test_attention_rejects_bad_arguments(L):
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    spa = L.ei_sparse_prefill_attn
    assert spa(FAKE, FAKE, FAKE, d, t, 0.088, FAKE, FAKE, 0, FAKE, None, 0, None) == -2
    assert spa(FAKE, FAKE, FAKE, d, t, 0.088, None, FAKE, 10, FAKE, None, 0, None) == -1
    assert spa(FAKE, FAKE, FAKE, eb.Dims(1, 4, 1, 1024, 96), t, 0.088, FAKE, FAKE, 10, FAKE,
               None, 0, None) == -3
    # the scheduling workspace: EI_ATTN_WORKSPACE_BYTES, 16-byte aligned
    assert spa(FAKE, FAKE, FAKE, d, t, 0.088, FAKE, FAKE, 10, FAKE, FAKE,
               eb.ATTN_WORKSPACE_BYTES - 1, None) == -4
    assert spa(FAKE, FAKE, FAKE, d, t, 0.088, FAKE, FAKE, 10, FAKE, _off(FAKE, 4),
               eb.ATTN_WORKSPACE_BYTES, None) == -3
    assert L.ei_dense_prefill_attn(FAKE, FAKE, None, d, 0.088, 1, FAKE, None) == -1
    assert L.ei_dense_prefill_attn(FAKE, FAKE, FAKE, eb.Dims(1, 5, 2, 64, 128), 0.088, 1, FAKE,
                                   None) == -2
    assert L.ei_dense_prefill_attn(FAKE, FAKE, FAKE, d, float("nan"), 1, FAKE, None) == -2


def test_prefill_rejects_bad_arguments(L):
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    p = eb.budget_params(base_budget=256)
    km = L.ei_kmax(t, p)
    ws = L.ei_prefill_workspace_bytes(d, t)
    assert ws > 0 and ws == L.ei_probe_workspace_bytes(d, t) + eb.ATTN_WORKSPACE_BYTES
    outs = (FAKE,) * 7
    call = L.ei_entropy_guided_prefill
    args = (FAKE, FAKE, FAKE, d, t, 1.0, p)
    assert call(*args, 5, km, 0.088, *outs, FAKE, ws, None) == -2
    assert call(*args, 0, km - 1, 0.088, *outs, FAKE, ws, None) == -2
    assert call(*args, 0, km, 0.088, *outs, FAKE, ws - 1, None) == -4
    assert call(*args, 0, km, 0.088, *outs, None, ws, None) == -4
    assert call(None, FAKE, FAKE, d, t, 1.0, p, 0, km, 0.088, *outs, FAKE, ws, None) == -1


def test_prefill_workspace_is_the_probe_workspace(L):
    """The one-call path runs the three stages over the whole layer, so its
    workspace is the whole problem's probe workspace followed by the
    attention's scheduling workspace."""
    t = eb.Tiling(128, 64)
    for n in (1024, 8192, 16384, 131072):
        d = eb.Dims(2, 32, 8, n, 128)
        pw = L.ei_probe_workspace_bytes(d, t)
        assert pw > 0 and pw % 256 == 0
        assert L.ei_prefill_workspace_bytes(d, t) == pw + eb.ATTN_WORKSPACE_BYTES


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU: --gpus above 1 (or a multi-rank launch)
    exits with status 2 and says why, before touching a device."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    for extra_env, args in (({}, ["--gpus", "2"]), ({"WORLD_SIZE": "2"}, [])):
        env = dict(os.environ, **extra_env)
        r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), *args],
                           capture_output=True, text=True, timeout=120, env=env, cwd=root)
        assert r.returncode == 2, (args, extra_env, r.stderr[-500:])
        assert "one GPU" in (r.stdout + r.stderr)


def test_binding_shape_checks():
    """The binding refuses tensors whose sizes differ from what the C ABI
    derives from q's shape and seq_len (a kernel would read past them)."""
    import pytest
    from paper_2606_09508_amd import binding as eb
    q = (1, 4, 128, 128)
    eb.check_qkv_shapes(q, (1, 2, 128, 128), (1, 2, 128, 128))
    for kb in [(2, 2, 128, 128), (1, 2, 64, 128), (1, 2, 128, 64), (1, 3, 128, 128),
               (1, 0, 128, 128), (1, 2, 128)]:
        with pytest.raises(ValueError):
            eb.check_qkv_shapes(q, kb)
    with pytest.raises(ValueError):
        eb.check_qkv_shapes(q, (1, 2, 128, 128), (1, 2, 127, 128))
    eb.check_score_shapes((1, 4, 8, 16), (1, 4, 8), 1024, 128, 64)
    eb.check_score_shapes((2, 4, 8, 16), (2, 4, 8), 1000, 128, 64)     # ragged tail
    for ls, en, n in [((1, 4, 8, 15), (1, 4, 8), 1024), ((1, 4, 8, 16), (1, 4, 7), 1024),
                      ((1, 4, 8, 16), (1, 4, 8), 1100), ((1, 4, 8, 16), (2, 4, 8), 1024),
                      ((4, 8, 16), (4, 8), 1024)]:
        with pytest.raises(ValueError):
            eb.check_score_shapes(ls, en, n, 128, 64)


def _off(p, n):
    return ctypes.c_void_p(p.value + n)


def test_misaligned_pointers_are_refused(L):
    """bf16 tensors and workspaces need 16-byte, fp32 / int32 arrays 4-byte
    alignment; anything else returns EI_ERR_UNSUPPORTED before a launch."""
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    need = L.ei_probe_workspace_bytes(d, t)
    probe = L.ei_entropy_probe
    assert probe(_off(FAKE, 2), FAKE, d, t, 1.0, FAKE, FAKE, FAKE, need, None) == -3
    assert probe(FAKE, _off(FAKE, 8), d, t, 1.0, FAKE, FAKE, FAKE, need, None) == -3
    assert probe(FAKE, FAKE, d, t, 1.0, _off(FAKE, 2), FAKE, FAKE, need, None) == -3
    assert probe(FAKE, FAKE, d, t, 1.0, FAKE, FAKE, _off(FAKE, 8), need, None) == -3
    p = eb.budget_params(base_budget=256)
    km = L.ei_kmax(t, p)
    sel = L.ei_select_blocks
    assert sel(_off(FAKE, 2), FAKE, d, t, p, km, FAKE, FAKE, FAKE, FAKE, None) == -3
    assert sel(FAKE, FAKE, d, t, p, km, FAKE, FAKE, _off(FAKE, 1), FAKE, None) == -3
    assert sel(FAKE, FAKE, d, t, p, km, _off(FAKE, 1), FAKE, FAKE, _off(FAKE, 3), None) == -3
    spa = L.ei_sparse_prefill_attn
    assert spa(FAKE, FAKE, _off(FAKE, 8), d, t, 0.088, FAKE, FAKE, km, FAKE, None, 0,
               None) == -3
    assert spa(FAKE, FAKE, FAKE, d, t, 0.088, FAKE, FAKE, km, _off(FAKE, 4), None, 0,
               None) == -3
    assert spa(FAKE, FAKE, FAKE, d, t, 0.088, _off(FAKE, 2), FAKE, km, FAKE, None, 0,
               None) == -3
    assert L.ei_dense_prefill_attn(FAKE, _off(FAKE, 2), FAKE, d, 0.088, 1, FAKE, None) == -3
    assert L.ei_dense_prefill_attn(FAKE, FAKE, FAKE, d, 0.088, 0, _off(FAKE, 8), None) == -3
    ws = L.ei_prefill_workspace_bytes(d, t)
    call = L.ei_entropy_guided_prefill
    outs = [FAKE] * 7
    assert call(FAKE, FAKE, _off(FAKE, 2), d, t, 1.0, p, 0, km, 0.088, *outs, FAKE, ws,
                None) == -3
    bad = list(outs)
    bad[4] = _off(FAKE, 2)   # block_idx
    assert call(FAKE, FAKE, FAKE, d, t, 1.0, p, 0, km, 0.088, *bad, FAKE, ws, None) == -3
    assert call(FAKE, FAKE, FAKE, d, t, 1.0, p, 0, km, 0.088, *outs, _off(FAKE, 8), ws,
                None) == -3


def test_sizes_whose_grids_overflow_are_refused(L):
    """B x Hq x ceil(N / 128) workgroups must fit in 31 bits (every launch's
    grid is bounded by it): larger problems are EI_ERR_SHAPE on the host."""
    t = eb.Tiling(128, 64)
    big = eb.Dims(1, 1 << 20, 1 << 10, 1 << 20, 128)      # 2^20 heads x 2^13 tiles
    assert L.ei_num_segments(big, t) == -1
    assert L.ei_probe_workspace_bytes(big, t) == 0
    assert L.ei_entropy_probe(FAKE, FAKE, big, t, 1.0, FAKE, FAKE, FAKE, 1 << 30, None) == -2
    assert L.ei_dense_prefill_attn(FAKE, FAKE, FAKE, big, 0.088, 1, FAKE, None) == -2
    assert L.ei_sparse_prefill_attn(FAKE, FAKE, FAKE, big, t, 0.088, FAKE, FAKE, 98, FAKE,
                                    None, 0, None) == -2
    ok = eb.Dims(1, 1 << 17, 1 << 10, 1 << 20, 128)       # 2^17 x 2^13 = 2^30 workgroups
    assert L.ei_num_segments(ok, t) == (1 << 20) // 128


def test_gqa_union_attention_limits(L):
    """The GQA-union mode holds the merged list in LDS: kmax <= 128 and
    C_B <= 8192, else EI_ERR_UNSUPPORTED; otherwise it validates like
    ei_sparse_prefill_attn."""
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    call = L.ei_sparse_prefill_attn_gqa_union
    assert call(FAKE, FAKE, FAKE, d, t, 0.088, FAKE, FAKE, 129, FAKE, None) == -3
    long = eb.Dims(1, 4, 1, 8192 * 64 + 64, 128)
    assert call(FAKE, FAKE, FAKE, long, t, 0.088, FAKE, FAKE, 98, FAKE, None) == -3
    assert call(FAKE, FAKE, FAKE, d, t, 0.088, FAKE, FAKE, 0, FAKE, None) == -2
    assert call(FAKE, FAKE, None, d, t, 0.088, FAKE, FAKE, 98, FAKE, None) == -1
    assert call(FAKE, FAKE, _off(FAKE, 8), d, t, 0.088, FAKE, FAKE, 98, FAKE, None) == -3
    assert call(FAKE, FAKE, FAKE, eb.Dims(0, 4, 1, 1024, 128), t, 0.088, None, None, 98, None,
                None) == 0


def test_bench_counter_figures_are_scoped():
    """bench.py takes traffic / matrix-busy figures from the committed counter
    summaries only for the workload and seed they were collected on, and only
    while their recorded kernel-source hash is the current one."""
    import os
    import shutil
    import sys
    import tempfile
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import bench
    for wl in (("c1", 0), ("c3", 1), ("c5", 0)):
        assert bench.read_traffic(wl) is None
        assert bench.read_counter_file(bench.SQ_FILE, "mfma_busy_fraction", wl) is None
    # a summary whose hash is not the current source's is ignored
    with tempfile.TemporaryDirectory() as d:
        p = os.path.join(d, "t.txt")
        shutil.copy(bench.TRAFFIC_FILE, p)
        good = bench.read_counter_file(p, "hbm_bytes_per_launch")
        txt = open(p).read()
        cur = bench.sources_hash(bench.ATTN_SOURCES)
        assert (good is not None) == (f"attn_source_hash: {cur}" in txt)
        open(p, "w").write(txt.replace("attn_source_hash:", "attn_source_hash: 0"))
        assert bench.read_counter_file(p, "hbm_bytes_per_launch") is None


BAD_SCALES = (0.0, -0.088, float("inf"), float("-inf"), float("nan"))


@pytest.mark.parametrize("scale", BAD_SCALES)
def test_attention_refuses_non_positive_or_non_finite_scales(L, scale):
    """The kernels mask scores before scaling and take the maximum of the raw
    scores, which is the maximum of the scaled ones only for a positive scale:
    every attention entry point (and the one-call path) refuses a
    softmax_scale that is not finite and > 0 before any launch."""
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    km = 98
    assert L.ei_sparse_prefill_attn(FAKE, FAKE, FAKE, d, t, scale, FAKE, FAKE, km, FAKE,
                                    None, 0, None) == -2
    assert L.ei_sparse_prefill_attn_gqa_union(FAKE, FAKE, FAKE, d, t, scale, FAKE, FAKE, km,
                                              FAKE, None) == -2
    for causal in (0, 1):
        assert L.ei_dense_prefill_attn(FAKE, FAKE, FAKE, d, scale, causal, FAKE, None) == -2
    p = eb.budget_params()
    ws = L.ei_prefill_workspace_bytes(d, t)
    assert L.ei_entropy_guided_prefill(FAKE, FAKE, FAKE, d, t, 1.0, p, 0, L.ei_kmax(t, p), scale,
                                       *(FAKE,) * 7, FAKE, ws, None) == -2


@pytest.mark.parametrize("ps", (float("inf"), float("-inf"), float("nan")))
def test_probe_refuses_non_finite_probe_scale(L, ps):
    d, t = eb.Dims(1, 4, 1, 1024, 128), eb.Tiling(128, 64)
    need = L.ei_probe_workspace_bytes(d, t)
    assert L.ei_entropy_probe(FAKE, FAKE, d, t, ps, FAKE, FAKE, FAKE, need, None) == -2
    p = eb.budget_params()
    ws = L.ei_prefill_workspace_bytes(d, t)
    assert L.ei_entropy_guided_prefill(FAKE, FAKE, FAKE, d, t, ps, p, 0, L.ei_kmax(t, p), 0.088,
                                       *(FAKE,) * 7, FAKE, ws, None) == -2


def test_noalloc_prefill_refusals(L):
    """ei_entropy_guided_prefill_noalloc validates like the workspace entry
    point and refuses, before touching a device, a problem whose probe
    workspace exceeds its static scratch array (128 MiB)."""
    t, p = eb.Tiling(128, 64), eb.budget_params()
    km = L.ei_kmax(t, p)
    call = L.ei_entropy_guided_prefill_noalloc
    outs = (FAKE,) * 7
    big = eb.Dims(1, 64, 8, 262144, 128)   # the Llama-3-70B layer at 256k
    assert L.ei_prefill_workspace_bytes(big, t) > 128 << 20
    assert call(FAKE, FAKE, FAKE, big, t, 1.0, p, 0, km, 0.088, *outs, None) == -4
    for fits in (eb.Dims(1, 32, 8, 131072, 128), eb.Dims(1, 64, 8, 131072, 128)):
        assert L.ei_prefill_workspace_bytes(fits, t) <= 128 << 20   # the 8B and 70B layers
    d = eb.Dims(1, 32, 8, 131072, 128)
    assert call(FAKE, FAKE, FAKE, d, t, 1.0, p, 0, km, 0.0, *outs, None) == -2
    assert call(None, FAKE, FAKE, d, t, 1.0, p, 0, km, 0.088, *outs, None) == -1
    assert call(FAKE, FAKE, FAKE, eb.Dims(1, 4, 1, 1024, 96), t, 1.0, p, 0, km, 0.088, *outs,
                None) == -3
    assert call(None, None, None, eb.Dims(0, 4, 1, 1024, 128), t, 1.0, p, 0, km, 0.088,
                *(None,) * 7, None) == 0

@pytest.mark.parametrize("n,tiling", [(1000, (128, 64)), (1, (128, 64)), (130, (256, 128)),
                                      (131071, (128, 64))])
def test_ragged_sequence_lengths_are_accepted(L, n, tiling):
    """N need not be a multiple of L_S or L_B (a deliberate superset of the
    boundary's shape rule): the shape checks pass and the call stops at the
    next check, the missing workspace, before anything is launched."""
    d, t = eb.Dims(1, 4, 1, n, 128), eb.Tiling(*tiling)
    assert L.ei_num_segments(d, t) == -(-n // t.seg_len)
    assert L.ei_num_blocks(d, t) == -(-n // t.block_len)
    assert L.ei_probe_workspace_bytes(d, t) > 0
    assert L.ei_entropy_probe(FAKE, FAKE, d, t, 1.0, FAKE, FAKE, FAKE, 0, None) == -4
    p = eb.budget_params()
    km = L.ei_kmax(t, p)
    assert L.ei_entropy_guided_prefill(FAKE, FAKE, FAKE, d, t, 1.0, p, 0, km, 0.088,
                                       *((FAKE,) * 7), FAKE, 0, None) == -4


def test_fused_probe_select_refusals(L):
    """ei_probe_select_fused validates like the probe and the selection
    together, needs the probe workspace plus 64 bytes per (b, h, s), and
    refuses rows of more than 2048 past blocks (its LDS rows), all before
    anything is launched."""
    t, p = eb.Tiling(128, 64), eb.budget_params()
    km = L.ei_kmax(t, p)
    call = L.ei_probe_select_fused
    outs = (FAKE,) * 5
    for n in (1024, 131072):
        d = eb.Dims(2, 32, 8, n, 128)
        need = L.ei_probe_select_workspace_bytes(d, t)
        assert need >= L.ei_probe_workspace_bytes(d, t) + 2 * 32 * (n // 128) * 64
        assert call(FAKE, FAKE, d, t, 1.0, p, 0, km, *outs, FAKE, need - 1, None) == -4
        assert call(FAKE, FAKE, d, t, 1.0, p, 0, km, *outs, None, need, None) == -4
    d = eb.Dims(1, 4, 1, 1024, 128)
    need = L.ei_probe_select_workspace_bytes(d, t)
    assert call(None, FAKE, d, t, 1.0, p, 0, km, *outs, FAKE, need, None) == -1
    assert call(FAKE, FAKE, d, t, 1.0, p, 0, km, FAKE, FAKE, None, FAKE, FAKE, FAKE, need,
                None) == -1
    assert call(FAKE, FAKE, d, t, 1.0, p, 3, km, *outs, FAKE, need, None) == -2
    assert call(FAKE, FAKE, d, t, 1.0, p, 0, km - 1, *outs, FAKE, need, None) == -2
    assert call(FAKE, FAKE, d, t, float("nan"), p, 0, km, *outs, FAKE, need, None) == -2
    assert call(FAKE, FAKE, eb.Dims(1, 4, 1, 1024, 96), t, 1.0, p, 0, km, *outs, FAKE, need,
                None) == -3
    assert call(None, None, eb.Dims(0, 4, 1, 1024, 128), t, 1.0, p, 0, km, *(None,) * 5, None,
                0, None) == 0
    # the longest supported rows: 2048 past blocks (the last segment at 131072 + 128 tokens
    # with L_S = 128, L_B = 64 has 2048; one token more starts a segment with 2050)
    for n, tl, ok in ((131072 + 128, (128, 64), True), (131072 + 129, (128, 64), False),
                      (262144 + 256, (256, 128), True), (262144 + 257, (256, 128), False)):
        dd, tt = eb.Dims(1, 4, 1, n, 128), eb.Tiling(*tl)
        kk = L.ei_kmax(tt, p)
        need = L.ei_probe_select_workspace_bytes(dd, tt)
        st = call(FAKE, FAKE, dd, tt, 1.0, p, 0, kk, *outs, FAKE, 0, None)
        assert st == (-4 if ok else -3), (n, tl, st)
