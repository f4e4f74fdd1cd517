"""The paper's constants against every place that defaults to them.

tests/golden/paper_constants.json holds each constant with the passage that
states it (App. B.1, B.2, D.1.1, D.1.2, D.1.5, D.3).  The package's defaults
module, the binding's keyword defaults and the oracle's keyword defaults must
all equal those values, so a constant retyped wrong in any of them fails here.
"""
import inspect
import json
import os

import pytest

import oracle
from paper_2609_33570_amd import defaults as D

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def gold(key):
    ent = GOLD[key]
    assert ent["cite"], key
    return ent["value"]


def default_of(fn, name):
    return inspect.signature(fn).parameters[name].default


def test_fixture_entries_cited():
    keys = [k for k in GOLD if not k.startswith("_")]
    assert len(keys) == 11
    for k in keys:
        assert set(GOLD[k]) == {"value", "cite"} and GOLD[k]["cite"].strip(), k


@pytest.mark.parametrize("attr,key", [
    ("CLIP_EPS", "clip_eps"), ("KL_BETA", "kl_beta"), ("ADV_EPS", "adv_eps"),
    ("EPS_ALPHA", "eps_alpha"), ("EPS_REL", "eps_rel"), ("EPS_NUM", "eps_num"),
    ("N_B", "n_b"), ("N_DELTA", "n_delta"), ("LORA_RANK", "lora_rank"),
    ("LORA_ALPHA", "lora_alpha"), ("TOP_FRAC", "top_frac")])
def test_package_defaults(attr, key):
    assert getattr(D, attr) == gold(key)


def test_lora_scale():
    # App. D.1.1: the adapter output is scaled by alpha / r
    assert D.LORA_SCALE == gold("lora_alpha") / gold("lora_rank") == 2.0


@pytest.mark.parametrize("fn,param,key", [
    ("grpo_advantages", "adv_eps", "adv_eps"), ("grpo_coeffs", "clip_eps", "clip_eps"),
    ("grpo_coeffs", "adv_eps", "adv_eps"), ("grpo_loss", "clip_eps", "clip_eps"),
    ("unit_exposure_risk", "eps_alpha", "eps_alpha"), ("unit_exposure_risk", "eps_rel", "eps_rel"),
    ("allocate", "n_b", "n_b"), ("allocate", "n_d", "n_delta"),
    ("grad_rel_err", "eps_num", "eps_num"), ("update_sparsity", "top_frac", "top_frac")])
def test_oracle_defaults(fn, param, key):
    assert default_of(getattr(oracle, fn), param) == gold(key)


@pytest.mark.parametrize("fn,param,key", [
    ("hilore_allocate_workspace_bytes", "n_b", "n_b"),
    ("hilore_allocate_workspace_bytes", "n_d", "n_delta"),
    ("hilore_grad_rel_err", "eps_num", "eps_num")])
def test_binding_defaults(fn, param, key):
    from paper_2609_33570_amd import hilore
    assert default_of(getattr(hilore, fn), param) == gold(key)
