"""The C ABI on the CPU: libo5.so loads, exports every function include/o5.h
declares, and rejects bad arguments on the host before anything is enqueued
(no GPU needed: these calls fail validation before any HIP call)."""
import ctypes
import os
import re

import pytest

from paper_1912_06680_amd import o5

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "o5.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(o5_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(o5.LIB_PATH):
        pytest.skip("libo5.so not built")
    return o5.lib()


def test_header_declares_the_binding_table():
    assert _declared_functions() == sorted(o5.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert o5.o5_version() == 100
    assert o5.o5_status_str(0).startswith("O5_OK")
    assert o5.o5_status_str(5).startswith("O5_E_WORKSPACE")


def test_host_validation_errors(lib):
    L = lib
    # NULL pointers are rejected with O5_E_NULL
    st = L.o5_gae(16, 8, None, None, None, 0.99, 0.95, None, None, None)
    assert st == 1 and "NULL" in o5.o5_last_error()
    # shapes
    assert L.o5_gae(0, 8, 16, 16, 16, 0.99, 0.95, 16, 16, None) == 2
    assert L.o5_segments_to_samples(10, 2, 3, 16, 16, 16, 16, 16, 16, None) == 2
    # misaligned pointer
    assert L.o5_gae(16, 8, 0x1001, 16, 16, 0.99, 0.95, 16, 16, None) == 4
    # argument range
    assert L.o5_gae(16, 8, 16, 16, 16, 1.5, 0.95, 16, 16, None) == 7
    hp = o5.AdamHp(1e-3, 0.9, 0.999, 1e-8, 5.0)
    assert L.o5_adam_step(10, 16, 16, 16, 16, None, hp, 0, None) == 7
    # dtype and LSTM shapes
    assert L.o5_lstm_fwd(9, 1, 1, 64, 64, *([16] * 11), 1 << 20, None) == 3
    assert L.o5_lstm_fwd(0, 1, 1, 60, 64, *([16] * 11), 1 << 20, None) == 2
    # B is bounded by the cell kernels' grids (32 rows per block, y < 65535)
    assert L.o5_lstm_fwd_workspace_bytes(1, 1, 32767 * 64, 64, 64) > 0
    assert L.o5_lstm_fwd_workspace_bytes(1, 1, 32767 * 64 + 1, 64, 64) == 0
    assert L.o5_lstm_bptt_workspace_bytes(0, 1, 32767 * 64 + 1, 64, 64) == 0
    # workspace too small
    need = L.o5_lstm_fwd_workspace_bytes(1, 16, 8, 64, 128)
    assert need > 0
    assert L.o5_lstm_fwd(1, 16, 8, 64, 128, *([16] * 11), need - 1, None) == 5
    # reward post-processing: shapes, argument ranges, workspace
    rhp = o5.RewardHp(0.3, 0.6, 10.0, 1e-8)
    assert L.o5_reward_process(0, 4, 16, None, 16, rhp, 16, 16, 16, 1 << 20, None) == 2
    assert L.o5_reward_process(4, 4, 16, None, None, rhp, 16, 16, 16, 1 << 20, None) == 1
    assert L.o5_reward_process(4, 4, 16, 0x1008, 16, rhp, 16, 16, 16, 1 << 20, None) == 4
    assert L.o5_reward_process(4, 4, 16, None, 16, o5.RewardHp(1.5, 0.6, 10.0, 1e-8), 16, 16, 16, 1 << 20,
                               None) == 7
    assert L.o5_reward_process(4, 4, 16, None, 16, o5.RewardHp(0.3, 0.6, 0.0, 1e-8), 16, 16, 16, 1 << 20,
                               None) == 7
    need = L.o5_reward_process_workspace_bytes(4, 4)
    assert need > 0
    assert L.o5_reward_process(4, 4, 16, None, 16, rhp, 16, 16, 16, need - 1, None) == 5
    # input side: teams of five, widths multiple of 64
    assert L.o5_prelstm_fwd(1, 2, 7, 64, 64, 16, 16, 16, 16, 16, None) == 2
    assert L.o5_prelstm_fwd(1, 2, 10, 64, 96, 16, 16, 16, 16, 16, None) == 2
    assert L.o5_prelstm_fwd(5, 2, 10, 64, 64, 16, 16, 16, 16, 16, None) == 3
    assert L.o5_obs_normalize(0, 10, 6, 16, 16, 5.0, 1e-8, 16, 16, 1 << 20, None) == 2
    assert L.o5_obs_normalize(0, 10, 8, 16, 16, 0.0, 1e-8, 16, 16, 1 << 20, None) == 7
    # surgery: shrinking is not a widening; folding keeps at least one input
    assert L.o5_surgery_widen(64, 64, 9, 32, 64, 16, None, None, 16, 16, 16, 0.01, 1, None) == 2
    assert L.o5_surgery_widen(64, 64, 9, 64, 128, 16, None, None, 16, 16, 16, -1.0, 1, None) == 7
    assert L.o5_surgery_widen(64, 64, 9, 64, 128, None, None, None, 16, 16, 16, 0.01, 1, None) == 1
    assert L.o5_surgery_fold_input(64, 64, 9, 64, 16, 16, None, None, 16, 16, 16, None) == 2
    assert L.o5_param_count(4096, 4096, 75) == 134541387
    # heads
    heads = (ctypes.c_int * 2)(3, 0)
    assert L.o5_ppo_loss_grad_workspace_bytes(0, 8, 64, 2, heads, None) == 0
    assert "head_sizes[1]" in o5.o5_last_error()


def test_factored_calls_validate_on_the_host(lib):
    L = lib
    heads = (ctypes.c_int * 4)(30, 8, 32, 4)
    assert L.o5_ppo_head_grad_ld(4096, 4, heads, None) == 256
    u = o5.UnitHead(1, 128, 16, 16, 16, 16, 16)
    assert L.o5_ppo_head_grad_ld(4096, 4, heads, ctypes.byref(u)) == 512
    assert L.o5_ppo_head_grad_ld(4096, 4, None, None) == 0
    need = L.o5_ppo_loss_grad_workspace_bytes(1, 2048, 4096, 4, heads, None)
    hp = o5.PpoHp(0.2, 1.0, 0.01)
    # h, Wp, bp, act, logp_old, adv, ret; no head mask, availability or unit
    # head (a host pointer); stats, P, W
    args = [2048, 4096, 4, heads] + [16] * 7 + [None, None, None] + [hp, 16, 16, 16]
    # fp32 is refused; ld must be the heads' value
    assert L.o5_ppo_loss_grad_factored(0, *args, 256, 16, 16, 16, need, None) == 3
    assert L.o5_ppo_loss_grad_factored(1, *args, 320, 16, 16, 16, need, None) == 2
    assert "o5_ppo_head_grad_ld" in o5.o5_last_error()
    bneed = L.o5_lstm_bptt_workspace_bytes(1, 16, 8, 64, 128)
    bargs = [16, 8, 64, 128] + [16] * 11
    assert L.o5_lstm_bptt_factored(0, *bargs, 256, *([16] * 6), 16, bneed, None) == 3
    assert L.o5_lstm_bptt_factored(1, *bargs, 100, *([16] * 6), 16, bneed, None) == 2
    assert L.o5_lstm_bptt_factored(1, *bargs, 256, *([16] * 6), 16, bneed - 1, None) == 5


def test_workspace_queries_are_positive(lib):
    for dt in (0, 1):
        assert o5.o5_lstm_fwd_workspace_bytes(dt, 16, 2048, 4096, 4096) > 0
        assert o5.o5_lstm_bptt_workspace_bytes(dt, 16, 2048, 4096, 4096) > 0
        assert o5.o5_ppo_loss_grad_workspace_bytes(dt, 32768, 4096, (30, 8, 32, 4)) > 0
        assert o5.o5_policy_sample_workspace_bytes(dt, 4096, 4096, (30, 8, 32, 4)) > 0
    u = o5.UnitHead(1, 128, 16, 16, 16, 16, 16)
    base = o5.o5_ppo_loss_grad_workspace_bytes(1, 32768, 4096, (30, 8, 32, 4))
    assert o5.o5_ppo_loss_grad_workspace_bytes(1, 32768, 4096, (30, 8, 32, 4), u) > base
    assert o5.o5_policy_sample_workspace_bytes(1, 4096, 4096, (30, 8, 32, 4), u) > 0
    assert o5.o5_ppo_loss_grad_workspace_bytes(1, 64, 64, (3, 4), o5.UnitHead(2, 16, 16, 16, 16, 16, 16)) == 0
    assert o5.o5_reward_process_workspace_bytes(256, 13107) > 0
    assert o5.o5_reward_process_workspace_bytes(0, 1) == 0


def test_binding_arity_matches_header():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    found = 0
    for m in re.finditer(r"\b(o5_[a-z0-9_]+)\s*\(([^;{]*?)\)\s*;", text):
        name, args = m.group(1), m.group(2).strip()
        n = 0 if args in ("void", "") else args.count(",") + 1
        assert len(o5._SIGS[name][1]) == n, name
        found += 1
    assert found == len(o5.EXPORTED)
