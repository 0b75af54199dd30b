"""Pins for oracle.layout against the paper's worked examples."""
import json
import os
from types import SimpleNamespace as NS

import numpy as np
import pytest

import workloads
from oracle import layout as L

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_reordered_documents_example():
    g = _load("layout_reordered_docs.json")
    for q, order in g["orders"].items():
        lengths = [g["prefix_tokens"]] + [g["doc_tokens"]] * len(order)
        starts = L.layout(lengths)[1:]
        got = {doc: [s, s + g["doc_tokens"] - 1] for doc, s in zip(order, starts)}
        for doc, rng in g["stated"][q].items():
            assert got[doc] == rng, (q, doc)
        assert got == g["implied"][q]


def test_kv_bytes_per_token_example():
    g = _load("kv_bytes_per_token.json")
    per_rank = L.kv_bytes_per_token(g["L"], g["H_kv"], g["d_h"], g["w"], g["TP"])
    assert per_rank == g["bytes_per_token_per_rank"]
    assert per_rank * g["TP"] == g["bytes_per_token_all_ranks"]


@pytest.mark.parametrize("n,B,pages", [(1, 16, 1), (16, 16, 1), (17, 16, 2),
                                       (512, 16, 32), (64, 16, 4), (255, 16, 16)])
def test_pages_for(n, B, pages):
    assert L.pages_for(n, B) == pages


def _unit(pos, n, res, r, retain=0, pages=None):
    return NS(unit_id=0, position=pos, n_tokens=n, residency=res,
              n_recompute=r, retain=retain,
              pool_pages=np.arange(L.pages_for(n, 16)) if pages is None else pages)


def test_sets_partition_the_prompt():
    req = NS(prompt_len=10 + 40 + 30 + 25 + 7,
             text_segs=[(0, 10), (105, 7)],
             units=[_unit(10, 40, L.HIT, 4), _unit(50, 30, L.MISS, 4),
                    _unit(80, 25, L.HIT, 100)])
    L.check_tiling(req)
    comp = set(L.compute_positions(req).tolist())
    gath = {p for _, _, p in L.gather_tokens(req)}
    assert comp.isdisjoint(gath)
    assert comp | gath == set(range(req.prompt_len))
    # text, whole miss unit, first 4 of the first hit, all of the short hit
    assert len(comp) == 10 + 4 + 30 + 25 + 7


def test_tiling_violations_raise():
    base = dict(prompt_len=30, text_segs=[(0, 10)])
    with pytest.raises(ValueError):
        L.check_tiling(NS(**base, units=[_unit(11, 20, L.HIT, 0)]))   # gap
    with pytest.raises(ValueError):
        L.check_tiling(NS(**base, units=[_unit(9, 21, L.HIT, 0)]))    # overlap
    with pytest.raises(ValueError):
        L.check_tiling(NS(**base, units=[_unit(10, 19, L.HIT, 0)]))   # short


def test_retain_block_addressing():
    pages = np.array([7, 3, 11], dtype=np.int32)
    req = NS(prompt_len=40, text_segs=[], units=[_unit(0, 40, L.MISS, 0, 1, pages)])
    toks = L.retain_tokens(req, 16)
    assert [(t[3], t[4]) for t in toks[:2]] == [(7, 0), (7, 1)]
    assert (toks[16][3], toks[16][4]) == (3, 0)
    assert (toks[39][3], toks[39][4]) == (11, 7)


def test_generated_workloads_are_contiguous_layouts():
    for name in ["tiny", "small_bf16", "small_f32", "rag8b"]:
        wl = workloads.generate(name)
        for req in wl.requests:
            L.check_tiling(req)
            segs = L.segments(req)
            assert [s for _, s, _, _ in segs] == L.layout([n for _, _, n, _ in segs])
