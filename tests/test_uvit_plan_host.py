"""Host checks of the transformer-model planning inputs: the op layout and
long skips of the UViT and Hunyuan-DiT-like models, and the memory model's
parameter count against the stage library's own parameter layout."""

import pytest

from paper_2606_19163_amd import configs
from paper_2606_19163_amd import tstage as TS
from paper_2606_19163_amd import uvit_plan as U


@pytest.mark.parametrize("name", sorted(U.MODELS))
def test_ops_and_mirror_skips(name):
    m = U.MODELS[name]
    names, kinds, skips = U.uvit_ops(m["n_in"], m["mid"])
    n_in = m["n_in"]
    assert len(names) == len(kinds) == 2 * n_in + (1 if m["mid"] else 0)
    assert kinds.count("dec") == n_in
    assert len(skips) == n_in
    for i, (a, b) in enumerate(skips):
        assert names[a] == f"in{i}" and names[b] == f"out{n_in - 1 - i}"
        assert kinds[a] == "enc" and kinds[b] == "dec"
    # nested: the first encoder block feeds the last decoder block, and every
    # skip's span contains the spans of the skips inside it
    spans = sorted(skips)
    for (a0, b0), (a1, b1) in zip(spans, spans[1:]):
        assert a0 < a1 < b1 < b0


@pytest.mark.parametrize("name", sorted(U.MODELS))
def test_param_bytes_match_stage_layout(name):
    """Two bytes per parameter of one encoder block plus one decoder block
    equal two bytes per parameter of a 1 + 1 transformer stage."""
    m = U.MODELS[name]
    d = configs._tstage(1, m["tokens"], m["width"], m["heads"], 1, 1)
    d["mlp"] = m["mlp"]
    st = TS.TStage(d, dry_run=True)
    assert U.param_bytes("enc", m) + U.param_bytes("dec", m) == 2.0 * st.n_params


def test_activation_model_counts_kept_tensors():
    m = U.MODELS["hdit"]
    C, R, L = m["width"], m["mlp"] * m["width"], m["tokens"]
    assert U.act_bytes_per_sample("enc", m) == 2.0 * L * (8 * C + 2 * R)
    assert U.act_bytes_per_sample("dec", m) - U.act_bytes_per_sample("enc", m) == 2.0 * L * C
    assert U.out_bytes_per_sample(m) == 2.0 * L * C
