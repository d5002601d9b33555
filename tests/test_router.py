"""The prompt-complexity router (SS III-B) and the placement plan (SS III-C):
host logic, no GPU.  The features are checked on hand-counted prompts, the
score for monotonicity in each feature, the classes against the thresholds
and the long-prompt rule, calibration against the shares it is given, and
the placement against the byte counts of each variant."""
import dataclasses
import math

import pytest

from paper_2609_21704_amd import synth
from paper_2609_21704_amd.configs import CONFIGS, HEAD_DIM
from paper_2609_21704_amd.engine import cache_bytes, placement, weight_bytes
from paper_2609_21704_amd.router import PAPER_MIX, Features, Router, features, hash_tokenize, score


def test_hash_tokenizer():
    ids = hash_tokenize("Explain the harvest, please!", 151936)
    # Explai n | the | harves t | , | please | !  (words cut into pieces of six characters)
    assert len(ids) == 8
    assert all(0 <= t < 151936 for t in ids)
    assert ids == hash_tokenize("Explain the harvest, please!", 151936)
    assert hash_tokenize("the the", 1000)[0] == hash_tokenize("the the", 1000)[1]
    # FNV-1a of "a" (32 bit) is 0xE40C292C
    assert hash_tokenize("a", 1 << 32)[0] == 0xE40C292C
    assert hash_tokenize("", 10) == []


def test_features_hand_counted():
    f = features("Name the river.")
    assert f.tokens == 4
    assert f.syntax == pytest.approx(math.log2(3))  # three words, no clause
    assert f.entities == 0.0                          # "Name" opens the sentence
    text = "When did Maribeth Oduya visit Port Celestine in 1907, and why?"
    f = features(text)
    # 11 words; "When" subordinates (1), one comma (1/2); entities: Maribeth Oduya Port Celestine 1907
    assert f.syntax == pytest.approx(math.log2(11) + 1.5)
    assert f.entities == pytest.approx(5 / 11)
    assert f.tokens == len(hash_tokenize(text, 151936))
    # two sentences: the syntax term is their mean; bracket nesting counts its depth
    f = features("Compute f(g(x)) now. Then stop.")
    s1 = math.log2(5) + 2   # Compute f g x now: depth 2
    s2 = math.log2(2)
    assert f.syntax == pytest.approx((s1 + s2) / 2)
    # acronyms, inner capitals, inner dots and digits are entity-like; a sentence-initial capital is not
    f = features("Ask NASA about iPhone sales in Q3 via v2.5 docs.")
    assert f.entities == pytest.approx(4 / 10)  # ten words, four entity-like
    assert features("", tokens=0) == Features(0, 0.0, 0.0)
    assert features("whatever text", tokens=77).tokens == 77


def test_score_is_monotone_in_each_feature():
    base = Features(tokens=40, syntax=3.0, entities=0.1)
    s0 = score(base)
    assert score(dataclasses.replace(base, tokens=41)) > s0
    assert score(dataclasses.replace(base, syntax=3.5)) > s0
    assert score(dataclasses.replace(base, entities=0.2)) > s0
    # the reference point of every term is 1
    assert score(Features(512, 8.0, 0.3)) == pytest.approx(1.0)
    assert score(Features(0, 0.0, 0.0)) == 0.0


def test_classes_and_long_prompts():
    r = Router(low=0.3, high=0.6, long_tokens=1000)
    assert r.classify(Features(4, 1.0, 0.0)) == "int4"
    assert r.classify(Features(60, 3.0, 0.1)) == "fp8"
    assert r.classify(Features(400, 9.0, 0.4)) == "f16"
    assert r.classify(Features(1000, 0.0, 0.0)) == "f16"   # long context: full precision
    assert r.classify(Features(999, 0.0, 0.0)) != "f16"
    # a prompt said twice has the same sentences and density and twice the tokens:
    # it never routes to a lighter variant
    order = {"int4": 0, "fp8": 1, "f16": 2}
    for t in synth.prompt_texts(200, 3):
        assert order[r.route(t + " " + t)] >= order[r.route(t)]
    with pytest.raises(ValueError):
        Router(low=0.7, high=0.5)


def test_calibration_hits_the_shares():
    texts = synth.prompt_texts(1000, 8)
    r = Router().calibrate(texts)
    counts = {c: 0 for c in ("int4", "fp8", "f16")}
    for t in texts:
        counts[r.route(t)] += 1
    # exact on the calibration set up to prompts of equal score
    assert abs(counts["int4"] - 280) <= 2 and abs(counts["f16"] - 200) <= 2
    # close on a fresh set from the same mix
    fresh = synth.prompt_texts(2000, 9)
    share = sum(r.route(t) == "int4" for t in fresh) / 2000
    assert abs(share - PAPER_MIX[0]) < 0.04
    # degenerate shares
    r0 = Router().calibrate(texts, (0.0, 1.0, 0.0))
    assert all(r0.route(t) == "fp8" for t in texts)
    r1 = Router().calibrate(texts, (1.0, 0.0, 0.0))
    assert all(r1.route(t) == "int4" for t in texts)
    with pytest.raises(ValueError):
        Router().calibrate(texts, (0.5, 0.6, 0.0))


def test_default_thresholds_are_the_calibrated_ones():
    r = Router().calibrate(synth.prompt_texts(2000, 5))
    assert (round(r.low, 2), round(r.high, 2)) == (Router().low, Router().high)


def test_weight_and_cache_bytes():
    cfg = CONFIGS[2]  # 7B: 28 layers, hidden 3584, intermediate 18944, 28 / 4 heads, vocab 151936
    w = weight_bytes(cfg)
    H, I, V, L = 3584, 18944, 151936, 28
    per_layer = (28 * 128 + 2 * 4 * 128) * H + H * 28 * 128 + 2 * I * H + H * I
    nk = L * per_layer + V * H
    assert w["f16"] == 2 * nk + V * H * 2 + (2 * L + 1) * H * 2 + L * (28 + 8) * 128 * 2
    assert w["int4"] == nk // 2 + 4 * nk // 128
    rows = L * (28 * 128 + 2 * 4 * 128 + H + 2 * I + H) + V
    assert w["fp8"] == nk + 4 * rows
    assert 15.2e9 < w["f16"] < 15.3e9 and 3.7e9 < w["int4"] < 3.8e9
    assert cache_bytes(cfg, L, 4, 2048) == 2 * L * 4 * 4 * 2048 * HEAD_DIM * 2


def test_placement():
    cfg = CONFIGS[2]
    L, B, cap = 28, 4, 1024
    w = weight_bytes(cfg)
    c1 = cache_bytes(cfg, L, B, cap)
    full = placement(cfg, 288e9, B, cap, 4)
    assert full["resident"] == ["f16", "int4", "fp8"]
    assert full["route_to"] == {"int4": "int4", "fp8": "fp8", "f16": "f16"}
    # room for the parent and the INT4 draft only: FP8 requests go to INT4
    need = w["f16"] + c1 + w["int4"] + 2 * c1
    p = placement(cfg, need / 0.9 + 1e6, B, cap, 4)
    assert p["resident"] == ["f16", "int4"]
    assert p["route_to"] == {"int4": "int4", "fp8": "int4", "f16": "f16"}
    # room for the parent alone: everything decodes directly
    p = placement(cfg, (w["f16"] + c1) / 0.9 + 1e6, B, cap, 4)
    assert p["resident"] == ["f16"]
    assert set(p["route_to"].values()) == {"f16"}
    with pytest.raises(MemoryError):
        placement(cfg, w["f16"], B, cap, 4)
    # 32B: both drafts beside the parent in one GPU's HBM
    assert placement(CONFIGS[4], 288e9, 1, 2048, 6)["resident"] == ["f16", "int4", "fp8"]
