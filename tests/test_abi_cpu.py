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
                                 "emb_dim", "clip"])
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
    with pytest.raises(V.VflError) as e:
        V.vfl_workspace_size(a, b, t, o)
    assert e.value.status == V.VFL_E_INVALID
