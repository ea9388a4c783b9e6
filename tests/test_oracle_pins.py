"""The oracle against what the paper and the mathematics fix (CPU only)."""
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd.inputs import layer_group_count
from tests import oracle_pins as P

SCORE_CHECKS = [P.check_closed_form, P.check_denominator_is_previous, P.check_joint_mean,
                P.check_zero_change, P.check_eps_in_denominator, P.check_scale_invariance,
                P.check_exact_rational]


@pytest.mark.parametrize("check", SCORE_CHECKS, ids=lambda f: f.__name__)
def test_score_pins(check):
    check(O.layer_update_score)


@pytest.mark.parametrize("check", [P.check_ge_threshold, P.check_delta_in_fp64, P.check_k0_extremes,
                                   P.check_record_format,
                                   P.check_capacity, P.check_restore_errors,
                                   P.check_accum_equals_snapshot_first_step, P.check_resync, P.check_call_order_errors,
                                   P.check_record_format_weights_only, P.check_fused_step_rules,
                                   P.check_snapshot_partial_pack_refresh, P.check_layout_validation,
                                   P.check_unpacked_selection_blocks],
                         ids=lambda f: f.__name__)
def test_state_pins(check):
    check(O.LayerCheckOracle)


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
def test_staleness_period(mode):
    P.check_staleness_period(O.LayerCheckOracle, mode)


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
def test_irregular_steps(mode):
    P.check_irregular_steps(O.LayerCheckOracle, mode)


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
def test_zero_layer(mode):
    P.check_zero_layer(O.LayerCheckOracle, mode)


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
def test_rebase(mode):
    P.check_rebase(O.LayerCheckOracle, mode)


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
def test_stats_invariants(mode):
    P.check_stats_invariants(O.LayerCheckOracle, mode)


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
def test_restore_roundtrip(mode):
    P.check_restore_roundtrip(O.LayerCheckOracle, mode)


def test_bf16_round():
    """Section 4.1's bf16 weight copy: round to nearest, ties to even, against
    hand-worked bit patterns and torch's independent conversion."""
    P.check_bf16_round(O.bf16_round)


def test_fourteen_bytes_per_param():
    P.check_fourteen_bytes_per_param()


# Public architecture hyper-parameters of the three models in Table 1:
# (hidden, ffn, blocks, vocab, q heads, kv heads, qkv bias, tied lm_head)
TABLE1_MODELS = {
    "qwen2.5-7b": (3584, 18944, 28, 152064, 28, 4, True, False),
    "qwen2.5-3b": (2048, 11008, 36, 151936, 16, 2, True, True),
    "llama3.2-1b": (2048, 8192, 16, 128256, 32, 8, False, True),
}


def _table1_rows():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "table1_default_rows.txt")
    rows = []
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            name, n, writes, dirs, gb = line.split()
            rows.append((name, int(n), int(writes), int(dirs), float(gb)))
    return rows


@pytest.mark.parametrize("row", _table1_rows(), ids=lambda r: r[0])
def test_table1_layer_counts_and_record_size(row):
    """Table 1 (Section 4.3) Default rows: N = B + 3 untied / B + 2 tied
    (Section 2.2); every full checkpoint writes all N groups; and the mean
    full-checkpoint size equals the records of every layer at 14 bytes per
    parameter (bf16 copy + fp32 master + m + v, Section 4.1) within 0.2%."""
    from paper_2609_27193_amd.inputs import _decoder_layers
    name, n_layers, writes, dirs, mean_gb = row
    hidden, ffn, blocks, vocab, nq, nkv, bias, tied = TABLE1_MODELS[name]
    N = layer_group_count(blocks, tied)
    assert N == n_layers
    assert writes == dirs * N
    layers = _decoder_layers(hidden, ffn, blocks, vocab, nq, nkv, qkv_bias=bias, tied=tied)
    assert len(layers) == N
    total = sum(O.record_bytes([t.numel for t in l.tensors], 2, True) for l in layers)
    assert abs(total / 1e9 - mean_gb) / mean_gb < 2e-3, (total / 1e9, mean_gb)


def test_oracle_validation():
    from tests._helpers import HostLayout
    lay = HostLayout([[4], [4]], seed=0)
    with pytest.raises(O.OracleError) as e:
        O.LayerCheckOracle(lay.segs[::-1], 2, O.DT_BF16, True, O.MODE_ACCUM, [1e-3] * 2, 4)
    assert e.value.code == O.LC_ERR_INVALID_ARG
    orc = O.LayerCheckOracle(lay.segs, 2, O.DT_BF16, True, O.MODE_SNAPSHOT, [1e-3] * 2, 4)
    with pytest.raises(O.OracleError) as e:
        orc.score(1)  # base version not yet packed in SNAPSHOT mode
    assert e.value.code == O.LC_ERR_BAD_STATE
    orc.pack(0, 1 << 30)
    with pytest.raises(O.OracleError):
        orc.score(0)  # not after t_base
    orc.score(1)
    with pytest.raises(O.OracleError) as e:
        orc.select(1, 0.0)
    assert e.value.code == O.LC_ERR_INVALID_ARG
    with pytest.raises(O.OracleError) as e:
        orc.select(2, 1.0)
    assert e.value.code == O.LC_ERR_BAD_STATE
