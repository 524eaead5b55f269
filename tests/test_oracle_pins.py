"""The oracle against its pins (CPU only)."""
import numpy as np
import pytest

import oracle
from oracle import attention as oatt
from tests import oracle_pins as P


def test_switch_golden():
    P.pin_switch_golden(oracle.switch)


def test_switch_index_loops():
    P.pin_switch_index_loops(oracle.switch, oracle.switch_index_map)


def test_switch_round_trip():
    P.pin_switch_round_trip(oracle.switch, oracle.unswitch)


def test_switch_b1_is_transpose():
    P.pin_switch_b1_transpose(oracle.switch)


def test_switch_bits_and_copy():
    P.pin_switch_bits_and_copy(oracle.switch)


def test_switch_nrank_simulation():
    P.pin_switch_nrank_simulation(oracle.switch, oracle.exchange_unpack)


def test_switch_k3_index_loops():
    P.pin_switch_k3_index_loops(oracle.switch)


def test_switch_k3_unit_dim():
    P.pin_switch_k3_unit_dim(oracle.switch)


def test_switch_nrank_simulation_k3():
    P.pin_switch_nrank_simulation_k3(oracle.switch, oracle.exchange_unpack)


def test_split_gather():
    P.pin_split_gather(oracle.split, oracle.gather)


def test_switch_is_gather_then_split():
    P.pin_switch_is_gather_then_split(oracle.switch, oracle.exchange_unpack, oracle.split,
                                      oracle.gather)


def test_switch_rejects_bad_args():
    x = np.zeros((1, 4, 6, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.switch(x, 1, 2, 4)          # 6 % 4 != 0
    with pytest.raises(ValueError):
        oracle.switch(x[0], 1, 2, 1)       # not 4-D
    with pytest.raises(ValueError):
        oracle.switch(x, 0, 2, 1)
    with pytest.raises(ValueError):
        oracle.switch(np.zeros((1, 2, 2, 2, 2, 2)), 1, 2, 1)       # K = 4
    with pytest.raises(ValueError):
        oracle.switch(np.zeros((1, 2, 2, 2, 2)), 1, 4, 1)          # 4 is C for K = 3
    with pytest.raises(ValueError):
        oracle.split(x, 2, 4, 0)                                    # 6 % 4 != 0
    with pytest.raises(ValueError):
        oracle.split(x, 2, 2, 2)                                    # rank out of range


@pytest.mark.parametrize("pin", [P.pin_attention_brute, P.pin_attention_l1_is_v,
                                 P.pin_attention_zero_q_mean, P.pin_attention_two_keys_closed_form,
                                 P.pin_attention_rows_stochastic, P.pin_attention_hard_max,
                                 P.pin_attention_permutations, P.pin_attention_scale_default])
def test_attention(pin):
    pin(oracle.attention)


def test_spatial_temporal_units():
    P.pin_spatial_temporal_units(oracle.spatial_attention, oracle.temporal_attention,
                                 oracle.temporal_attention_strided, oracle.switch)


def test_layernorm():
    P.pin_layernorm(oracle.layernorm)


def test_linear():
    P.pin_linear(oracle.linear)


def test_gelu():
    P.pin_gelu(oracle.gelu)


def test_relu():
    P.pin_relu(oracle.relu)


def test_block_post_ln_relu():
    P.pin_block_post_ln_relu(oracle.st_block, oracle.layernorm, oracle.linear, oracle.relu,
                             oracle.switch, oracle.BLOCK_POST_LN, oracle.BLOCK_RELU)


def test_block_identities():
    P.pin_block_identities(oracle.st_block, oracle.layernorm, oracle.linear, oracle.gelu,
                           oracle.switch)


def test_block_t1_s1():
    P.pin_block_t1_s1(oracle.st_block, oracle.layernorm, oracle.linear, oracle.gelu)


def test_block_sharded_equals_unsharded():
    P.pin_block_sharded_equals_unsharded(oracle.st_block, oracle.layernorm, oracle.linear,
                                         oracle.gelu, oracle.switch, oracle.exchange_unpack,
                                         oracle.spatial_attention, oracle.temporal_attention)


def test_tiny_chain():
    P.pin_tiny_chain(oracle.tiny_chain, oracle.st_block)


def test_block_no_mlp_ln_flag():
    rng = np.random.default_rng(3)
    C, F, H = 8, 8, 2
    x = rng.standard_normal((1, 2, 3, C))
    p = {n: rng.standard_normal(s) * 0.3 for n, s in
         (("wqkv_s", (C, 3 * C)), ("wo_s", (C, C)), ("wqkv_t", (C, 3 * C)), ("wo_t", (C, C)),
          ("w1", (C, F)), ("w2", (F, C)))}
    a = oracle.st_block(x, p, H)
    b = oracle.st_block(x, p, H, flags=oracle.BLOCK_NO_MLP_LN)
    zc = np.zeros((F, C))
    base = oracle.st_block(x, dict(p, w2=zc), H)
    assert np.allclose(b, base + oracle.linear(oracle.gelu(oracle.linear(base, p["w1"])), p["w2"]))
    assert not np.allclose(a, b)


def test_attention_bwd_finite_differences():
    P.pin_attention_bwd_fd(oracle.attention, oracle.attention_bwd)


def test_attention_bwd_invariants():
    P.pin_attention_bwd_invariants(oracle.attention_bwd)


def test_attention_lse():
    P.pin_attention_lse(oracle.attention_lse)


def test_attention_bwd_units():
    P.pin_attention_bwd_units(oracle.attention_bwd, oracle.attention_bwd_units,
                              oracle.attention_lse_units, oracle.attention_lse,
                              oracle.attention_delta_units, oracle.attention)


# ---- block backward
from oracle import block_bwd as OB  # noqa: E402

BWD_FLAGS = [0, oracle.BLOCK_NO_MLP_LN, oracle.BLOCK_POST_LN, oracle.BLOCK_POST_LN | oracle.BLOCK_RELU,
             oracle.BLOCK_RELU | oracle.BLOCK_NO_MLP_LN]


def test_linear_bwd():
    P.pin_linear_bwd(oracle.linear, OB.linear_bwd)


def test_layernorm_bwd():
    P.pin_layernorm_bwd(oracle.layernorm, OB.layernorm_bwd)


def test_gelu_relu_bwd():
    P.pin_gelu_bwd(oracle.gelu, OB.gelu_bwd, oracle.relu, OB.relu_bwd)


def test_block_bwd_finite_differences():
    P.pin_block_bwd_fd(oracle.st_block, OB.st_block_bwd, BWD_FLAGS)


def test_block_bwd_matches_autograd():
    P.pin_block_bwd_autograd(OB.st_block_bwd, BWD_FLAGS)


def test_attention_grouped():
    P.pin_attention_grouped(oracle.attention_grouped, oracle.spatial_attention, oracle.attention)


def test_attention_grouped_bwd():
    P.pin_attention_grouped_bwd(oracle.attention_grouped, oracle.attention_grouped_bwd,
                                oracle.attention_bwd_units)
