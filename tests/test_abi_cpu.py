"""Host-side checks of the C-ABI library (no GPU): it loads, exports every
symbol include/vfl.h declares, validates configurations, and its pure host
scheduler equals the oracle's integer schedule."""
import os
import re

import pytest

import vfl_synth as S
from oracle import schedule

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def V():
    from paper_2510_12494_amd import vfl
    return vfl


def _declared():
    text = open(os.path.join(ROOT, "include", "vfl.h")).read()
    return sorted(set(re.findall(r"^\s*(?:vfl_status|const char\*)\s+(vfl_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol(V):
    names = _declared()
    assert len(names) >= 16
    lib = V.library()
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(V.EXPORTS)


@pytest.mark.parametrize("s", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("n_groups", [1, 5, 9])
def test_host_schedule_equals_oracle(V, s, n_groups):
    for t in range(n_groups + s):
        assert V.vfl_schedule_tick(t, s, n_groups) == schedule.tick_record(t, s, n_groups)


def test_schedule_rejects_bad_arguments(V):
    with pytest.raises(V.VflError):
        V.vfl_schedule_tick(0, 5, 3)
    with pytest.raises(V.VflError):
        V.vfl_schedule_tick(-1, 1, 3)


def test_workspace_size_for_every_workload(V):
    from paper_2510_12494_amd.session import bottom_spec, top_spec, opts
    sizes = {}
    for name in S.ALL:
        w = S.get(name)
        sizes[name] = V.vfl_workspace_size(bottom_spec(w.A), bottom_spec(w.B), top_spec(w.top), opts(w))
        assert sizes[name] > 0
    # a workspace scales with rows per tick and the channel depth s + 1
    assert sizes["hetero"] > sizes["dense_tabular"]
    w = S.get("dense_tabular")
    w2 = w.replace(staleness=4)
    a = V.vfl_workspace_size(bottom_spec(w.A), bottom_spec(w.B), top_spec(w.top), opts(w))
    b = V.vfl_workspace_size(bottom_spec(w2.A), bottom_spec(w2.B), top_spec(w2.top), opts(w2))
    assert b > a


@pytest.mark.parametrize("bad", ["staleness", "top_logit", "a_width", "no_hidden", "replicas",
                                 "emb_dim", "clip", "layers", "a_plus_top"])
def test_invalid_configurations_are_rejected(V, bad):
    from paper_2510_12494_amd.session import bottom_spec, top_spec, opts
    w = S.get("dense_tabular")
    a, b, t, o = bottom_spec(w.A), bottom_spec(w.B), top_spec(w.top), opts(w)
    if bad == "staleness":
        o.staleness = 5
    elif bad == "top_logit":
        t.widths[t.n_layers - 1] = 2
    elif bad == "a_width":
        a.widths[a.n_layers - 1] = 12
    elif bad == "no_hidden":
        t.n_layers = 1
        t.widths[0] = 1
    elif bad == "replicas":
        o.replicas = 9
    elif bad == "emb_dim":
        b.n_cat, b.vocab, b.emb_dim = 2, 10, 6
    elif bad == "clip":
        o.flags = V.VFL_CLIP_EMB
        o.clip_c = 0.0
    elif bad == "layers":
        b.n_layers = V.VFL_MAX_LAYERS + 1
    elif bad == "a_plus_top":
        # A's layers and the top's hidden layers share one weight-gradient launch
        a.n_layers = 10
        for i in range(10):
            a.widths[i] = 16
        t.n_layers = 8
        for i in range(7):
            t.widths[i] = 16
        t.widths[7] = 1
    with pytest.raises(V.VflError) as e:
        V.vfl_workspace_size(a, b, t, o)
    assert e.value.status == V.VFL_E_INVALID


def test_create_failures_report_their_reason(V):
    """A rejected configuration leaves its reason in vfl_last_error(NULL)."""
    from paper_2510_12494_amd.session import bottom_spec, top_spec, opts
    w = S.get("dense_tabular")
    a, b, t, o = bottom_spec(w.A), bottom_spec(w.B), top_spec(w.top), opts(w)
    o.staleness = 5
    with pytest.raises(V.VflError) as e:
        V.vfl_workspace_size(a, b, t, o)
    assert "staleness" in str(e.value)
    o.staleness = 2
    assert V.vfl_workspace_size(a, b, t, o) > 0
    assert V.vfl_last_error(None) == ""


def _random_shape(rng, dtype):
    from vfl_synth.workloads import Workload, PartySpec, TopSpec
    def widths(n, last_mult):
        ws = [int(rng.integers(1, 300)) for _ in range(n)]
        ws[-1] = int(rng.integers(1, 40)) * last_mult
        return ws
    cat = bool(rng.integers(0, 2))
    deep = bool(rng.integers(0, 4) == 0)        # a quarter of the shapes up to 12 layers deep
    nl = lambda: int(rng.integers(1, 13 if deep else 4))
    A = PartySpec(dense=int(rng.integers(1, 90)), widths=widths(nl(), 8))
    B = PartySpec(dense=int(rng.integers(0 if cat else 1, 90)), widths=widths(nl(), 1),
                  n_cat=int(rng.integers(1, 4)) if cat else 0, vocab=50, emb_dim=4 * int(rng.integers(1, 5)))
    top = TopSpec(widths=[int(rng.integers(1, 300)) for _ in range(int(rng.integers(1, 3)))] + [1])
    extra = bool(rng.integers(0, 2))
    return Workload(name="shape", n_rows=1000, dtype=dtype, A=A, B=B, top=top,
                    batch=int(rng.integers(1, 3000)), staleness=int(rng.integers(0, 5)),
                    replicas=int(rng.integers(1, 5)), lr=0.01, clip=1.0 if extra else 0.0,
                    sigma=0.5 if extra else 0.0, clip_emb=extra, clip_grad=extra, noise_emb=extra,
                    noise_grad=extra)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_host_plan_covers_random_shapes(V, dtype):
    """The host plan checks every chain layer's LDS and RC layout against
    what the kernels touch; any shape within the documented limits must
    pass (a failure here is an internal layout error, reported by text)."""
    import numpy as np
    from paper_2510_12494_amd.session import bottom_spec, top_spec, opts
    rng = np.random.default_rng(7 if dtype == "f32" else 8)
    for _ in range(300):
        w = _random_shape(rng, dtype)
        try:
            n = V.vfl_workspace_size(bottom_spec(w.A), bottom_spec(w.B), top_spec(w.top), opts(w))
        except V.VflError as e:
            # only the LDS capacity may refuse a shape within the limits
            assert "exceed the LDS" in str(e), (w, str(e))
            continue
        assert n > 0


def test_binding_fails_loudly_without_the_library(tmp_path):
    """No fallback: importing the binding where libvfl.so is missing raises
    (checked in a child interpreter on a copy of the package without the
    library)."""
    import shutil
    import subprocess
    import sys
    pkg = os.path.join(ROOT, "paper_2510_12494_amd")
    dst = tmp_path / "paper_2510_12494_amd"
    shutil.copytree(pkg, dst, ignore=shutil.ignore_patterns("*.so", "*.so.tmp", "__pycache__", "csrc"))
    assert not list(dst.glob("*.so"))
    code = "import paper_2510_12494_amd.vfl"
    r = subprocess.run([sys.executable, "-c", code], cwd=tmp_path, capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "no fallback" in r.stderr
