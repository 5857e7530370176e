"""The per-model presets (Table 3 configurations with the layer counts of Table 2 and the head
dimensions of Table 5) against the bit rates the paper prints for them, through the library's
host-only rate function (eq. (1) and eq. (3))."""
import pytest

import paper_2603_27467_amd as tvq
from paper_2603_27467_amd import presets

from test_abi_host import _cfg

# Table 2 "best per-layer" angle bits, Table 5 K8V4-log totals (the cells that follow eq. (3)),
# Table 6 norm8 on Mistral-7B
TABLE2_ANGLE_BITS = {"tinyllama-1.1b": 3.34, "mistral-7b": 3.31, "smollm2-1.7b": 3.67,
                     "phi-1.5": 3.58, "stablelm-2-1.6b": 3.63, "starcoder2-3b": 3.45,
                     "olmo-1b": 3.28}
TABLE5_K8V4LOG_BITS = {"smollm2-1.7b": 7.67, "phi-1.5": 7.58, "stablelm-2-1.6b": 7.63,
                       "starcoder2-3b": 7.45, "olmo-1b": 7.28}


def _rate(table, d, accounting=0):
    t = [(c.n_k, c.n_v, c.norm_bits_k, c.norm_bits_v, c.norm_mode_k, c.norm_mode_v)
         for c in table]
    return tvq.tvq_bits_per_element_config(_cfg(tvq, t, len(t), 8, d), accounting)


@pytest.mark.parametrize("model", sorted(TABLE2_ANGLE_BITS))
def test_table3_presets_give_table2_angle_bits(model):
    table, d = presets.table3_preset(model, norms="fp32")
    assert len(table) == presets.TABLE3[model][0]
    # fp32 norms add 16 bits per element (section 3.1, "Rate accounting")
    assert abs(_rate(table, d) - 16.0 - TABLE2_ANGLE_BITS[model]) <= 0.005


@pytest.mark.parametrize("model", sorted(TABLE5_K8V4LOG_BITS))
def test_table3_presets_give_table5_totals(model):
    table, d = presets.table3_preset(model, norms="k8v4log")
    assert abs(_rate(table, d) - TABLE5_K8V4LOG_BITS[model]) <= 0.005


def test_norm8_mistral_total():
    table, d = presets.table3_preset("mistral-7b", norms="norm8")
    assert d == 128
    assert abs(_rate(table, d) - 7.81) <= 0.005


def test_builders():
    t = presets.early_boost(6, 2)
    assert [(c.n_k, c.n_v) for c in t] == [(256, 128)] * 2 + [(128, 64)] * 4
    assert all((c.norm_bits_k, c.norm_bits_v) == (8, 4) for c in t)
    sel = presets.boosted_table(8, [0, 1, 6, 7], early=(256, 128))
    assert [c.n_k for c in sel] == [256, 256, 128, 128, 128, 128, 256, 256]
    # phi-1.5 skips layers 8-15 (section 3.4)
    phi, _ = presets.table3_preset("phi-1.5")
    assert [c.n_k for c in phi[8:16]] == [128] * 8 and phi[16].n_k == 256
    with pytest.raises(KeyError):
        presets.table3_preset("gpt-2")
    with pytest.raises(ValueError):
        presets.early_boost(4, 5)
    with pytest.raises(ValueError):
        presets.boosted_table(4, [4])
