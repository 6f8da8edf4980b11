"""Pins of the oracle's footprint, working-set and capacity arithmetic against
numbers the paper prints (tests/golden/paper_closed_forms.json cites each)."""
import json
import os

import pytest

import oracle

GIB = 1 << 30


@pytest.fixture(scope="module")
def paper(golden_dir):
    return json.load(open(os.path.join(golden_dir, "paper_closed_forms.json")))


def test_beta_full_model(paper):
    for m in ("qwen3_coder_30b_a3b", "qwen25_coder_32b"):
        c = paper["beta_bf16_full_model"][m]
        assert oracle.beta_rank(c["layers"], c["head_dim"], c["elem_bytes"], c["kv_heads"], 1) \
            == c["bytes_per_token"]


def test_footprint_table(paper):
    t = paper["footprint_table"]
    for i, tp in enumerate(t["tp"]):
        moe = oracle.beta_rank(48, 128, 2, 4, tp)
        dense = oracle.beta_rank(64, 128, 2, 8, tp)
        assert moe == t["moe_kib_per_rank"][i] * 1024
        assert dense == t["dense_kib_per_rank"][i] * 1024
        assert moe * tp == t["moe_aggregate_kib"][i] * 1024
        assert dense * tp == t["dense_aggregate_kib"][i] * 1024


def test_chunk_and_gpu_capacity(paper):
    c = paper["chunk_bytes_per_rank"]
    assert c["chunk_tokens"] * oracle.beta_rank(48, 128, 2, 4, 8) == c["mib"] << 20
    g = paper["gpu_kv_capacity_h20"]
    assert round(g["tokens"] * g["beta_rank"] / GIB, 2) == g["gib_2dp"]


def test_working_set_scale(paper):
    w = paper["working_set"]
    for case in w["cases"]:
        ws = oracle.working_set_bytes(case["A"], w["mean_prompt"], w["beta_rank"])
        assert round(ws / GIB, 1) == case["gib_1dp"]
        if "gib_2dp" in case:
            assert round(ws / GIB, 2) == case["gib_2dp"]
    ws16 = oracle.working_set_bytes(16, w["mean_prompt"], w["beta_rank"])
    for cap, val in zip(w["gamma_H"]["capacities_gib"], w["gamma_H"]["values"]):
        ndp = len(str(val).split(".")[1])
        assert round(ws16 / (cap * GIB), ndp) == val
    gG = w["gamma_G"]
    assert round(gG["A"] * w["mean_prompt"] / gG["K_G"], 2) == gG["value_2dp"]
    p = paper["working_set_planning"]
    a, b = p["cases"]
    assert round(oracle.working_set_bytes(a["agents"], a["context"], p["beta_rank"]) / GIB, 1) == a["gib_1dp"]
    assert round(oracle.working_set_bytes(b["agents"], b["context"], p["beta_rank"]) / GIB) == b["gib"]


def test_tier_chunks(paper):
    t = paper["tier_chunks"]
    for cap, kh in zip(t["capacities_gib"], t["K_H"]):
        assert oracle.tier_chunks(cap * GIB, t["block_tokens"], t["beta_rank"]) == kh


def test_tier_capacity_in_slots_matches_K_H(paper):
    # one slot per 1,024-token chunk at 24 KiB/token: the tier's slot count is
    # the paper's K_H (one 1,024-token "page" of 48 layers, 1 head, d=128, bf16)
    t = paper["tier_chunks"]
    sh = oracle.make_shape(1, 48, 1024, 1, 128, 2)
    assert oracle.sizes(sh)["slot"] == t["block_tokens"] * t["beta_rank"]
    for cap, kh in zip(t["capacities_gib"], t["K_H"]):
        assert oracle.Tier(sh, cap * GIB).capacity == kh


def test_layout_sizes_of_the_workloads():
    # Qwen3-30B-A3B full model (48 layers, 4 heads, d=128, bf16), 16-token pages
    s = oracle.sizes(oracle.make_shape(20000, 48, 16, 4, 128, 2))
    assert s["piece"] == 32 * 1024 and s["page"] == 1536 * 1024 and s["slot"] == s["page"]
    assert s["page"] == 16 * oracle.beta_rank(48, 128, 2, 4, 1)
    # fp8 with a per-(layer, page, K/V) fp32 scale: 48*8 = 384 B trailer -> 512
    s = oracle.sizes(oracle.make_shape(8192, 48, 16, 4, 128, 1, True))
    assert s["piece"] == 16 * 1024 and s["trailer"] == 512 and s["slot"] == 768 * 1024 + 512
    assert s["scales"] == 48 * 8192 * 8


def test_heads_per_rank_round_up_when_tp_does_not_divide():
    # Eq. 1 takes ceil(H_kv / TP): 6 heads over 4 ranks leave 2 heads on some rank
    assert oracle.beta_rank(10, 64, 2, 6, 4) == 2 * 10 * 64 * 2 * 2
    assert oracle.beta_rank(10, 64, 2, 3, 2) == 2 * 10 * 64 * 2 * 2


def test_restore_cost_and_obr_on_h20(paper):
    # the paper's H20 numbers: 24 KiB per token at the median 26.6 GiB/s is
    # 0.86 us per token; 6.6 GFLOP per token on eight GPUs at 148 TFLOPS is
    # at least 5.6 us; so OBR for long prefixes is at least 0.84 (Eq. 2)
    h = paper["restore_cost_h20"]
    b_eff = h["restore_median_gib_s"] * GIB
    t_load = oracle.restore_time(1, h["beta_rank"], b_eff, 0.0)
    assert round(t_load * 1e6, 2) == h["restore_us_per_token_2dp"]
    t_pf = h["gflop_per_token"] * 1e9 / (h["gpus"] * h["peak_tflops_per_gpu"] * 1e12)
    assert round(t_pf * 1e6, 1) == h["prefill_bound_us_per_token_1dp"]
    lim = oracle.obr_limit(h["beta_rank"], b_eff, t_pf)
    assert lim > h["obr_limit_at_least"]
    # the paper's own rounding of the same bound: 1 - 0.86 / 5.6 > 0.84
    assert 1 - h["restore_us_per_token_2dp"] / h["prefill_bound_us_per_token_1dp"] > 0.84
    assert abs(lim - (1 - t_load / t_pf)) < 1e-12


def test_obr_definition_and_limit():
    # OBR(n) = 1 - (n beta / B + tau) / (n t_pf): zero when restoring costs as
    # much as recomputing, the limit from below as n grows, the limit itself
    # when tau = 0, and the fixed overhead amortized as tau / n
    beta, B, tau, t_pf = 24576.0, 50e9, 20e-6, 2e-6
    lim = oracle.obr_limit(beta, B, t_pf)
    assert abs(lim - (1 - beta / (B * t_pf))) < 1e-15
    prev = -1e9
    for n in (1, 10, 100, 1000, 10 ** 4, 10 ** 6):
        v = oracle.obr(n, beta, B, tau, t_pf)
        assert prev < v < lim
        assert abs((1 - v) * n * t_pf - oracle.restore_time(n, beta, B, tau)) < 1e-12
        prev = v
    assert abs(oracle.obr(10 ** 9, beta, B, tau, t_pf) - lim) < 1e-6
    assert abs(oracle.obr(7, beta, B, 0.0, t_pf) - lim) < 1e-15
    n_even = tau / (t_pf - beta / B)  # T_load(n) = T_rec(n)
    assert abs(oracle.obr(n_even, beta, B, tau, t_pf)) < 1e-12
