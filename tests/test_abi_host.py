"""C ABI on the CPU: every declared symbol is exported, host-side rules and
argument validation. Nothing here launches a kernel: each call below fails
host validation before any HIP call is made.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from ce_workloads import config_layout, build_layout, small_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ce_router.h")

ce = pytest.importorskip("paper_2608_29291_amd")

FAKE = 0x10000  # never dereferenced: validation fails first


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ce_[a-z_]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) == 24
    for n in names:
        assert hasattr(ce.lib, n), n
    assert set(names) == set(ce.EXPORTED)


def test_version_and_status_strings():
    assert "gfx950" in ce.ce_version()
    for code in (0, -1, -2, -3, -4):
        assert ce.lib.ce_status_string(code).startswith(b"CE_")


@pytest.mark.parametrize("keep", [0.0, 0.1, 0.25, 0.3, 0.35, 0.4, 0.5, 0.8, 0.95, 1.0,
                                  1e-30, 0.999999940395355, 0.3333333])
def test_num_keep_matches_oracle(keep):
    for n in [0, 1, 2, 7, 100, 729, 1000, 4096, 8192, 123457, 2 ** 31 - 1]:
        assert ce.ce_num_keep(keep, n) == oracle.num_keep(np.float32(keep), n), (keep, n)


def test_num_keep_rejects():
    assert ce.ce_num_keep(1.5, 10) == -1
    assert ce.ce_num_keep(-0.1, 10) == -1
    assert ce.ce_num_keep(float("nan"), 10) == -1
    assert ce.ce_num_keep(0.5, -1) == -1


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_kept_count_host_matches_oracle(i):
    offs, flags = build_layout(config_layout(i))
    keep = {1: 0.5, 2: 0.35, 3: 0.5, 4: 0.4, 5: 0.3}[i]
    logits = np.random.default_rng(i).standard_normal(len(flags)).astype(np.float32)
    sel = oracle.select(logits, flags, offs, np.float32(keep))
    assert ce.ce_kept_count_host(offs, flags, keep) == len(sel["kept_idx"])


def test_kept_count_host_rejects_bad_offsets():
    flags = np.zeros(10, np.uint8)
    assert ce.ce_kept_count_host(np.array([0, 5, 3, 10], np.int32), flags, 0.5) == -1
    assert ce.ce_kept_count_host(np.array([1, 10], np.int32), flags, 0.5) == -1
    assert ce.ce_kept_count_host(np.array([0, 9], np.int32), flags, 0.5) == -1


def _batch(B=2, T=100, keep=0.5, cap=100, t=FAKE):
    return ce.CEBatch(B, T, FAKE, FAKE, t, keep, cap)


def _scorer(d=256, r_c=64, r_e=32, n_seg=4, dtype=ce.CE_BF16):
    return ce.CEScorerW(d, r_c, r_e, n_seg, dtype, FAKE, None, FAKE, 0.0, FAKE, None, FAKE, None)


def _ffn(d=256, F=512, n_sets=1, dtype=ce.CE_BF16):
    w = ce.CEFFNW(d, F, n_sets, dtype)
    for s in range(min(n_sets, 2)):
        w.w_gate[s] = FAKE
        w.w_up[s] = FAKE
        w.w_down[s] = FAKE
    return w


def score(b, w, hidden=FAKE, logits=FAKE):
    return ce.lib.ce_score(ctypes.byref(b) if b is not None else None, hidden,
                           ctypes.byref(w) if w is not None else None, logits, None, None)


@pytest.mark.parametrize("mut,code", [
    (lambda b, w: (None, w), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (b, None), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (_batch(B=0), w), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (_batch(B=65536), w), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (_batch(T=-1), w), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (_batch(keep=1.5), w), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (_batch(keep=float("nan")), w), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (_batch(t=None), w), ce.CE_ERR_INVALID_ARG),
    (lambda b, w: (b, _scorer(d=100)), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (b, _scorer(dtype=7)), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (b, _scorer(r_c=48)), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (b, _scorer(r_c=0)), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (b, _scorer(r_c=512, r_e=32)), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (b, _scorer(n_seg=0)), ce.CE_ERR_UNSUPPORTED),
    (lambda b, w: (b, _scorer(n_seg=17)), ce.CE_ERR_UNSUPPORTED),
])
def test_score_validation(mut, code):
    b, w = mut(_batch(), _scorer())
    assert score(b, w) == code


def score_ws(b, w, hidden=FAKE, logits=FAKE, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = ce.lib.ce_workspace_size(ce.CE_WS_SCORE, ctypes.byref(b), 256, 0, ce.CE_BF16) if b else 0
    return ce.lib.ce_score_ws(ctypes.byref(b) if b is not None else None, hidden,
                              ctypes.byref(w) if w is not None else None, logits, None, ws, ws_bytes, None)


def test_score_ws_validation():
    """ce_score_ws: the scorer checks of ce_score, then the workspace (10
    fp32 partial logits per token, whatever the scorer picks)."""
    b, w = _batch(T=1000), _scorer()
    need = ce.lib.ce_workspace_size(ce.CE_WS_SCORE, ctypes.byref(b), 256, 0, ce.CE_BF16)
    assert need >= 10 * 1000 * 4
    assert score_ws(None, w) == ce.CE_ERR_INVALID_ARG
    assert score_ws(b, None) == ce.CE_ERR_INVALID_ARG
    assert score_ws(b, _scorer(d=100)) == ce.CE_ERR_UNSUPPORTED
    assert score_ws(b, w, logits=None) == ce.CE_ERR_INVALID_ARG
    assert score_ws(b, w, hidden=None) == ce.CE_ERR_INVALID_ARG
    assert score_ws(b, w, ws=None) == ce.CE_ERR_WORKSPACE
    assert score_ws(b, w, ws_bytes=need - 1) == ce.CE_ERR_WORKSPACE


def test_score_null_buffers():
    assert score(_batch(), _scorer(), hidden=None) == ce.CE_ERR_INVALID_ARG
    assert score(_batch(), _scorer(), logits=None) == ce.CE_ERR_INVALID_ARG
    w = _scorer()
    w.w1_core = None
    assert score(_batch(), w) == ce.CE_ERR_INVALID_ARG
    w = _scorer()
    w.w1_exp = None
    assert score(_batch(), w) == ce.CE_ERR_INVALID_ARG


def test_topk_validation_and_workspace():
    b = _batch()
    need = ce.lib.ce_workspace_size(ce.CE_WS_TOPK, ctypes.byref(b), 256, 512, ce.CE_BF16)
    assert need >= 256 and need % 256 == 0
    f = ce.lib.ce_topk_compact
    # workspace too small / missing / misaligned
    assert f(ctypes.byref(b), FAKE, None, 0, 0, FAKE, FAKE, None, None, FAKE, need - 1, None) == ce.CE_ERR_WORKSPACE
    assert f(ctypes.byref(b), FAKE, None, 0, 0, FAKE, FAKE, None, None, None, need, None) == ce.CE_ERR_WORKSPACE
    assert f(ctypes.byref(b), FAKE + 8, None, 0, 0, FAKE, FAKE, None, None, FAKE + 8, need, None) == ce.CE_ERR_WORKSPACE
    # null outputs
    assert f(ctypes.byref(b), FAKE, None, 0, 0, None, FAKE, None, None, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), FAKE, None, 0, 0, FAKE, None, None, None, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), None, None, 0, 0, FAKE, FAKE, None, None, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    # compact requested with a bad d / dtype / no hidden
    assert f(ctypes.byref(b), FAKE, FAKE, ce.CE_BF16, 100, FAKE, FAKE, None, FAKE, FAKE, need, None) == ce.CE_ERR_UNSUPPORTED
    assert f(ctypes.byref(b), FAKE, FAKE, 5, 256, FAKE, FAKE, None, FAKE, FAKE, need, None) == ce.CE_ERR_UNSUPPORTED
    assert f(ctypes.byref(b), FAKE, None, ce.CE_BF16, 256, FAKE, FAKE, None, FAKE, FAKE, need, None) == ce.CE_ERR_INVALID_ARG


def test_ffn_validation():
    b = _batch()
    f = ce.lib.ce_routed_ffn
    need = ce.lib.ce_workspace_size(ce.CE_WS_FFN, ctypes.byref(b), 256, 512, ce.CE_BF16)
    assert need >= 100 * 512 * 2
    assert f(ctypes.byref(b), FAKE, FAKE, FAKE, ctypes.byref(_ffn()), FAKE, FAKE, need - 256, None) == ce.CE_ERR_WORKSPACE
    assert f(ctypes.byref(b), FAKE, FAKE, FAKE, ctypes.byref(_ffn(F=100)), FAKE, FAKE, need, None) == ce.CE_ERR_UNSUPPORTED
    assert f(ctypes.byref(b), FAKE, FAKE, FAKE, ctypes.byref(_ffn(n_sets=3)), FAKE, FAKE, need, None) == ce.CE_ERR_UNSUPPORTED
    w = _ffn(n_sets=2)
    w.w_down[1] = None
    assert f(ctypes.byref(b), FAKE, FAKE, FAKE, ctypes.byref(w), FAKE, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), None, FAKE, FAKE, ctypes.byref(_ffn()), FAKE, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), FAKE, FAKE, None, ctypes.byref(_ffn()), FAKE, FAKE, need, None) == ce.CE_ERR_INVALID_ARG


def test_scatter_and_block_validation():
    b = _batch()
    assert ce.lib.ce_scatter_residual(ctypes.byref(b), FAKE, FAKE, FAKE, ce.CE_BF16, 72, FAKE, FAKE, None) == ce.CE_ERR_UNSUPPORTED
    assert ce.lib.ce_scatter_residual(ctypes.byref(b), FAKE, FAKE, None, ce.CE_BF16, 256, FAKE, FAKE, None) == ce.CE_ERR_INVALID_ARG
    fb = ce.lib.ce_routed_block
    need = ce.lib.ce_workspace_size(ce.CE_WS_BLOCK, ctypes.byref(b), 256, 512, ce.CE_BF16)
    sw, fw = _scorer(), _ffn()
    assert fb(ctypes.byref(b), FAKE, FAKE, ctypes.byref(sw), ctypes.byref(fw), None, None, None, FAKE, need - 256, None) == ce.CE_ERR_WORKSPACE
    assert fb(ctypes.byref(b), FAKE, FAKE, ctypes.byref(_scorer(d=512)), ctypes.byref(fw), None, None, None, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    assert fb(ctypes.byref(b), FAKE, FAKE, ctypes.byref(_scorer(dtype=ce.CE_F32)), ctypes.byref(fw), None, None, None, FAKE, need, None) == ce.CE_ERR_INVALID_ARG
    assert fb(ctypes.byref(b), None, FAKE, ctypes.byref(sw), ctypes.byref(fw), None, None, None, FAKE, need, None) == ce.CE_ERR_INVALID_ARG


def test_workspace_sizes_grow_with_capacity():
    small = _batch(cap=10)
    big = _batch(cap=1000)
    for which in (ce.CE_WS_FFN, ce.CE_WS_BLOCK):
        a = ce.lib.ce_workspace_size(which, ctypes.byref(small), 256, 512, ce.CE_BF16)
        c = ce.lib.ce_workspace_size(which, ctypes.byref(big), 256, 512, ce.CE_BF16)
        assert c - a >= 990 * 512 * 2
    assert ce.lib.ce_workspace_size(9, ctypes.byref(small), 256, 512, ce.CE_BF16) == 0
    assert ce.lib.ce_workspace_size(ce.CE_WS_BLOCK, ctypes.byref(small), 256, 512, 3) == 0


def test_host_logic_under_sanitizers(tmp_path):
    """Host-only build of the validation / keep-count code with ASan + UBSan (g++, no HIP)."""
    src = os.path.join(ROOT, "paper_2608_29291_amd", "csrc", "ce_host.cpp")
    drv = tmp_path / "drv.c"
    drv.write_text(r'''
#include <stdio.h>
#include <stdint.h>
#include "ce_router.h"
int main(void) {
  int32_t offs[4] = {0, 3, 3, 10};
  uint8_t flags[10] = {2, 0, 0, 0, 2, 0, 0, 0, 0, 0};
  int64_t kt = ce_kept_count_host(3, 10, offs, flags, 0.5f);
  int ok = (kt == 1 + 1 + 0 + 1 + 3) && ce_num_keep(0.35f, 729) == 256 && ce_num_keep(1.0f, 5) == 5
           && ce_num_keep(0.0f, 5) == 0 && ce_num_keep(1e-30f, 2147483647) == 1
           && ce_num_keep(2.0f, 5) == -1;
  ce_batch b = {2, 100, (const int32_t*)16, (const uint8_t*)16, 0, 0.5f, 50};
  size_t a = ce_workspace_size(CE_WS_BLOCK, &b, 256, 512, CE_BF16);
  ok = ok && a > 50 * 512 * 2 && (a % 256) == 0;
  printf("%s %lld %zu\n", ok ? "OK" : "FAIL", (long long)kt, a);
  return ok ? 0 : 1;
}
''')
    exe = tmp_path / "drv"
    cmd_cpp = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               f"-I{os.path.join(ROOT, 'include')}", "-c", src, "-o", str(tmp_path / "host.o")]
    cmd_c = ["gcc", "-O1", "-g", "-fsanitize=address,undefined", f"-I{os.path.join(ROOT, 'include')}",
             "-c", str(drv), "-o", str(tmp_path / "drv.o")]
    cmd_ld = ["g++", "-fsanitize=address,undefined", str(tmp_path / "host.o"), str(tmp_path / "drv.o"),
              "-o", str(exe)]
    for cmd in (cmd_cpp, cmd_c, cmd_ld):
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0 and r.stdout.startswith("OK"), r.stdout + r.stderr


def test_drop_stability_validation():
    b = _batch()
    st = lambda bb, tpt=FAKE, tpr=FAKE, jac=FAKE: ce.lib.ce_drop_stability(
        ctypes.byref(bb) if bb is not None else None, tpt, tpr, jac, None, None, None)
    assert st(None) == ce.CE_ERR_INVALID_ARG
    assert st(_batch(B=0)) == ce.CE_ERR_INVALID_ARG
    assert st(b, jac=None) == ce.CE_ERR_INVALID_ARG
    assert st(b, tpt=None) == ce.CE_ERR_INVALID_ARG
    assert st(b, tpr=None) == ce.CE_ERR_INVALID_ARG


def test_ffn_pruning_validation():
    b, w = _batch(), _ffn()
    assert ce.lib.ce_ffn_down_colnorms(None, FAKE, None) == ce.CE_ERR_INVALID_ARG
    assert ce.lib.ce_ffn_down_colnorms(ctypes.byref(w), None, None) == ce.CE_ERR_INVALID_ARG
    assert ce.lib.ce_ffn_down_colnorms(ctypes.byref(_ffn(F=100)), FAKE, None) == ce.CE_ERR_UNSUPPORTED
    need = ce.lib.ce_workspace_size(ce.CE_WS_FFN, ctypes.byref(b), 256, 512, ce.CE_BF16)

    def sal(bb=b, ww=w, act=FAKE, idx=FAKE, off=FAKE, norms=FAKE, mask=FAKE, delta=0.15, s=FAKE, lam=FAKE,
            ws=FAKE, ws_bytes=need):
        return ce.lib.ce_ffn_saliency(ctypes.byref(bb), act, idx, off, ctypes.byref(ww), norms, mask, delta,
                                      s, lam, None, ws, ws_bytes, None)
    assert sal(off=None) == ce.CE_ERR_INVALID_ARG
    assert sal(norms=None) == ce.CE_ERR_INVALID_ARG
    assert sal(mask=None) == ce.CE_ERR_INVALID_ARG
    assert sal(s=None) == ce.CE_ERR_INVALID_ARG
    assert sal(lam=None) == ce.CE_ERR_INVALID_ARG
    assert sal(act=None) == ce.CE_ERR_INVALID_ARG
    assert sal(delta=float("nan")) == ce.CE_ERR_INVALID_ARG
    assert sal(delta=float("inf")) == ce.CE_ERR_INVALID_ARG
    assert sal(ws=None) == ce.CE_ERR_WORKSPACE
    assert sal(ws_bytes=need - 1) == ce.CE_ERR_WORKSPACE
    assert sal(ww=_ffn(dtype=5)) == ce.CE_ERR_UNSUPPORTED

    def msk(bb=b, act=FAKE, off=FAKE, dtype=ce.CE_BF16, F=512, mask=FAKE, use=FAKE):
        return ce.lib.ce_ffn_mask_channels(ctypes.byref(bb), act, off, dtype, F, mask, use, None)
    assert msk(act=None) == ce.CE_ERR_INVALID_ARG
    assert msk(off=None) == ce.CE_ERR_INVALID_ARG
    assert msk(mask=None) == ce.CE_ERR_INVALID_ARG
    assert msk(use=None) == ce.CE_ERR_INVALID_ARG
    assert msk(F=100) == ce.CE_ERR_UNSUPPORTED
    assert msk(dtype=3) == ce.CE_ERR_UNSUPPORTED


def test_layer_gap_validation():
    b = _batch()

    def gap(bb=b, xi=FAKE, xo=FAKE, dtype=ce.CE_BF16, d=256, tp=FAKE, delta=0.004, cos=FAKE, ra=FAKE,
            rr=FAKE, g=FAKE):
        return ce.lib.ce_layer_gap(ctypes.byref(bb) if bb is not None else None, xi, xo, dtype, d, tp, delta,
                                   cos, ra, rr, g, None, None)
    assert gap(None) == ce.CE_ERR_INVALID_ARG
    assert gap(_batch(B=0)) == ce.CE_ERR_INVALID_ARG
    for k in ("xi", "xo", "tp", "cos", "ra", "rr", "g"):
        assert gap(**{k: None}) == ce.CE_ERR_INVALID_ARG, k
    assert gap(delta=float("nan")) == ce.CE_ERR_INVALID_ARG
    assert gap(d=100) == ce.CE_ERR_UNSUPPORTED
    assert gap(d=0) == ce.CE_ERR_UNSUPPORTED
    assert gap(dtype=9) == ce.CE_ERR_UNSUPPORTED


def _attn(**kw):
    f = dict(B=2, n_heads=12, n_kv_heads=2, head_dim=128, q_offsets=FAKE, kv_offsets=FAKE, q_capacity=100,
             kv_capacity=100, causal=1, scale=0.088, dtype=ce.CE_BF16)
    f.update(kw)
    return ce.CEAttn(**f)


@pytest.mark.parametrize("kw,ptrs,code", [
    ({}, {"q": None}, ce.CE_ERR_INVALID_ARG),
    ({}, {"o": None}, ce.CE_ERR_INVALID_ARG),
    ({}, {"k": None}, ce.CE_ERR_INVALID_ARG),
    ({}, {"v": None}, ce.CE_ERR_INVALID_ARG),
    ({"B": 0}, {}, ce.CE_ERR_INVALID_ARG),
    ({"n_heads": 12, "n_kv_heads": 5}, {}, ce.CE_ERR_INVALID_ARG),
    ({"n_kv_heads": 0}, {}, ce.CE_ERR_INVALID_ARG),
    ({"causal": 2}, {}, ce.CE_ERR_INVALID_ARG),
    ({"scale": float("nan")}, {}, ce.CE_ERR_INVALID_ARG),
    ({"scale": 0.0}, {}, ce.CE_ERR_INVALID_ARG),
    ({"scale": -0.1}, {}, ce.CE_ERR_INVALID_ARG),
    ({"q_offsets": None}, {}, ce.CE_ERR_INVALID_ARG),
    ({"kv_offsets": None}, {}, ce.CE_ERR_INVALID_ARG),
    ({"q_capacity": -1}, {}, ce.CE_ERR_INVALID_ARG),
    ({"head_dim": 64}, {}, ce.CE_ERR_UNSUPPORTED),
    ({"dtype": ce.CE_F32}, {}, ce.CE_ERR_UNSUPPORTED),
    ({"q_capacity": 1 << 20, "n_heads": 12}, {}, ce.CE_ERR_UNSUPPORTED),
])
def test_attention_validation(kw, ptrs, code):
    p = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE)
    p.update(ptrs)
    at = _attn(**kw)
    assert ce.lib.ce_routed_attention(ctypes.byref(at), p["q"], p["k"], p["v"], p["o"], None) == code
    assert ce.lib.ce_routed_attention(None, FAKE, FAKE, FAKE, FAKE, None) == ce.CE_ERR_INVALID_ARG


def tiling(B, T, d, r_c, r_e, dtype=ce.CE_BF16):
    out = (ctypes.c_int32 * 2)()
    r = ce.lib.ce_score_tiling(ctypes.byref(_batch(B=B, T=T)), ctypes.byref(_scorer(d=d, r_c=r_c, r_e=r_e,
                                                                                   dtype=dtype)), out)
    return r if r < 0 else (r, int(out[0]), int(out[1]))


@pytest.mark.parametrize("i,expect", [(1, (0, 32, 0)), (2, (0, 32, 0)), (3, (0, 128, 0)),
                                      (4, (1, 128, 128)), (5, (1, 128, 128))])
def test_score_tiling_of_named_workloads(i, expect):
    """Single-launch scorer with 32-token tiles for the tiny fp32 and the
    understanding workloads, with 128-token tiles for the generation workload
    (one round of workgroups instead of three), rank tiles of 128 x 128 for
    the 7B-width and MoT workloads (where 32-token tiles would each stream up
    to 2.8 MB of W1)."""
    from ce_workloads import config_params
    p = config_params(i)
    offs, flags = build_layout(config_layout(i))
    dt = ce.CE_F32 if i == 1 else ce.CE_BF16
    assert tiling(len(offs) - 1, len(flags), p["d"], p["r_c"], p["r_e"], dt) == expect


@pytest.mark.parametrize("T,r_c,r_e,expect", [(1024, 128, 32, (1, 64, 64)), (2176, 384, 96, (1, 64, 128)),
                                              (4224, 320, 32, (1, 128, 64)), (4224, 384, 96, (1, 128, 128)),
                                              (8320, 32, 64, (0, 128, 0)), (1024, 32, 32, (0, 32, 0))])
def test_score_tiling_shapes(T, r_c, r_e, expect):
    """Batch sizes that pick each scorer variant (the GPU parity tests use them)."""
    assert tiling(3, T, 192, r_c, r_e) == expect
    assert tiling(3, T, 192, r_c, r_e, dtype=ce.CE_F32) == (0, 32, 0)  # fp32: 32-token single launch


def test_score_tiling_validation():
    assert ce.lib.ce_score_tiling(None, ctypes.byref(_scorer()), None) == ce.CE_ERR_INVALID_ARG
    assert ce.lib.ce_score_tiling(ctypes.byref(_batch()), None, None) == ce.CE_ERR_INVALID_ARG
    assert tiling(0, 100, 256, 64, 32) == ce.CE_ERR_INVALID_ARG
    assert tiling(2, 100, 100, 64, 32) == ce.CE_ERR_UNSUPPORTED
    assert tiling(2, 100, 256, 64, 32) == (0, 32, 0)


# Partial-sum tiles the FFN workspace reserves for the split tail tiles of the
# two GEMM launches (the largest plan over gate/up, down and one or two weight
# sets), worked by hand from the plan's rule: per XCD (8) the items past full
# rounds of 32 run as S pieces each, when there are at most two full rounds.
# Understanding workload: down 108 tiles -> 14 per XCD, S = 2 (224 slots);
# two sets: 114 -> 15, S = 2 (240); gate/up 1260 / 1330 tiles: 4-5 full rounds,
# no split. Generation workload: gate/up 2380 tiles (9 rounds), down 204 (26 per
# XCD: S = 1), no split. 7B width: down 294 -> 37 = 32 + 5, S = 6 (240); MoT
# (two sets, the same tile counts): 240. fp32: none.
SPLIT_SLOTS = {1: 0, 2: 240, 3: 0, 4: 240, 5: 240}


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_gemm_split_workspace_of_named_workloads(i):
    from ce_workloads import config_params
    p = config_params(i)
    offs, flags = build_layout(config_layout(i))
    keep = {1: 0.5, 2: 0.35, 3: 0.5, 4: 0.4, 5: 0.3}[i]
    cap = ce.ce_kept_count_host(offs, flags, keep)
    dt = ce.CE_F32 if i == 1 else ce.CE_BF16
    elem = 4 if i == 1 else 2
    B, F = len(offs) - 1, p["F"]
    b = _batch(B=B, T=len(flags), keep=keep, cap=cap)
    need = ce.lib.ce_workspace_size(ce.CE_WS_FFN, ctypes.byref(b), p["d"], F, dt)
    al = lambda x: (max(x, 1) + 255) // 256 * 256
    slots = SPLIT_SLOTS[i]
    want = (al(16) + al(cap * 4) + al(4) + al(cap * F * elem)
            + (al(slots * 256 * 256 * 4) + 2 * al(256 * 4) if slots else 0)
            + al((16 * B * F + B * ((F + 255) // 256) * 2) * 4))
    assert need == want


def test_binding_rejects_host_tensors_before_any_call():
    """The binding checks what a pointer cannot carry (device, dtype, size,
    alignment) before calling the library; host tensors never reach it."""
    import torch
    wl = small_workload("und", seed=0, dtype="bf16", d=64, F=64, r_c=32, r_e=32)
    t = lambda x, dt=None: torch.from_numpy(np.ascontiguousarray(x)) if dt is None else \
        torch.from_numpy(np.ascontiguousarray(x)).to(dt)
    batch = ce.Batch(t(wl.seq_offsets), t(wl.flags), t(wl.t), float(wl.keep), wl.T)
    with pytest.raises(ValueError, match="GPU memory"):
        batch.c()
    sw = wl.scorer
    scorer = ce.Scorer(t(sw.w1_core, torch.bfloat16), t(sw.w2_core), t(sw.w1_exp, torch.bfloat16), t(sw.w2_exp))
    with pytest.raises(ValueError):
        scorer.c()
    with pytest.raises(ValueError):
        ce.ce_score(batch, t(wl.hidden, torch.bfloat16), scorer, torch.empty(wl.T))


def test_noalloc_topk_validation():
    """ce_topk_compact_noalloc rejects bad arguments and batches beyond its
    fixed scratch before any HIP call (so these run without a GPU)."""
    f = ce.lib.ce_topk_compact_noalloc
    b = _batch()
    assert f(None, FAKE, None, 0, 0, FAKE, FAKE, None, None, None, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), FAKE, None, 0, 0, FAKE, None, None, None, None, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), None, None, 0, 0, FAKE, FAKE, None, None, None, None) == ce.CE_ERR_INVALID_ARG
    assert f(ctypes.byref(b), FAKE, FAKE, ce.CE_BF16, 100, FAKE, FAKE, None, FAKE, None, None) == ce.CE_ERR_UNSUPPORTED
    big = _batch(B=65537, T=70000, cap=70000)
    assert f(ctypes.byref(big), FAKE, None, 0, 0, FAKE, FAKE, None, None, None, None) == ce.CE_ERR_UNSUPPORTED


def test_block_gap_validation():
    """ce_routed_block_gap rejects missing gap outputs, a non-finite delta and
    a workspace sized for ce_routed_block (CE_WS_BLOCK) before any launch."""
    f = ce.lib.ce_routed_block_gap
    b = _batch(cap=60)
    sw, fw = _scorer(), _ffn()
    need = ce.lib.ce_workspace_size(ce.CE_WS_BLOCK_GAP, ctypes.byref(b), 256, 512, ce.CE_BF16)
    small = ce.lib.ce_workspace_size(ce.CE_WS_BLOCK, ctypes.byref(b), 256, 512, ce.CE_BF16)
    assert need > small
    args = lambda **k: [ctypes.byref(b), FAKE, FAKE, ctypes.byref(sw), ctypes.byref(fw), None, None, None,
                        k.get("delta", 0.004), k.get("cos", FAKE), k.get("ra", FAKE), k.get("rr", FAKE),
                        k.get("g", FAKE), None, FAKE, k.get("ws", need), None]
    assert f(*args(cos=None)) == ce.CE_ERR_INVALID_ARG
    assert f(*args(ra=None)) == ce.CE_ERR_INVALID_ARG
    assert f(*args(g=None)) == ce.CE_ERR_INVALID_ARG
    assert f(*args(delta=float("nan"))) == ce.CE_ERR_INVALID_ARG
    assert f(*args(ws=small)) == ce.CE_ERR_WORKSPACE


def test_pruned_ffn_validation():
    """ce_routed_ffn_pruned rejects missing outputs, a non-finite delta, a
    channel split that is not whole 64-channel groups, fp32 and a workspace of
    the plain FFN kind before any launch."""
    f = ce.lib.ce_routed_ffn_pruned
    b = _batch(cap=60)
    fw = _ffn(d=256, F=512)
    need = ce.lib.ce_workspace_size(ce.CE_WS_FFN_PRUNED, ctypes.byref(b), 256, 512, ce.CE_BF16)
    plain = ce.lib.ce_workspace_size(ce.CE_WS_FFN, ctypes.byref(b), 256, 512, ce.CE_BF16)
    assert need > plain
    args = lambda **k: [ctypes.byref(b), FAKE, FAKE, FAKE, ctypes.byref(k.get("w", fw)), k.get("norms", FAKE),
                        k.get("n_keep", 384), k.get("delta", 0.15), FAKE, k.get("sal", FAKE), FAKE,
                        k.get("use", FAKE), FAKE, k.get("ws", need), None]
    assert f(*args(norms=None)) == ce.CE_ERR_INVALID_ARG
    assert f(*args(sal=None)) == ce.CE_ERR_INVALID_ARG
    assert f(*args(use=None)) == ce.CE_ERR_INVALID_ARG
    assert f(*args(delta=float("inf"))) == ce.CE_ERR_INVALID_ARG
    assert f(*args(n_keep=100)) == ce.CE_ERR_UNSUPPORTED
    assert f(*args(n_keep=576)) == ce.CE_ERR_UNSUPPORTED
    assert f(*args(w=_ffn(d=256, F=512, dtype=ce.CE_F32))) == ce.CE_ERR_UNSUPPORTED
    assert f(*args(ws=plain)) == ce.CE_ERR_WORKSPACE
