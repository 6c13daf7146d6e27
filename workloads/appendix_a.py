"""The tensor-contraction benchmark of Appendix A (Tables III and IV).

48 contractions in the paper's C-A-B encoding (Sec. 7.1: the index strings of
C, A and B, one character per index), each with the index extents the paper
uses in single precision (Table III) and in double precision (Table IV), and
whether the paper's LoG column has a result (a '-' there: Loops-over-GEMM is
not applicable to that contraction).  Shapes only: the inputs are synthetic
(seeded, U[-1,1]), alpha = 1, beta = 0.  The paper's timings are not used.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

from . import Workload

# (contraction, Table III extents, Table IV extents, LoG applicable)
TABLE: List[Tuple[str, Dict[str, int], Dict[str, int], bool]] = [
    ("abc-bda-dc", {"a": 384, "c": 24, "b": 384, "d": 384}, {"a": 312, "c": 24, "b": 312, "d": 312}, False),
    ("abc-dca-bd", {"a": 384, "c": 376, "b": 24, "d": 384}, {"a": 312, "c": 296, "b": 24, "d": 312}, True),
    ("abcd-dbea-ec", {"a": 96, "c": 24, "b": 84, "e": 96, "d": 96}, {"a": 72, "c": 24, "b": 72, "e": 72, "d": 72}, False),
    ("abcd-deca-be", {"a": 96, "c": 84, "b": 24, "e": 84, "d": 96}, {"a": 72, "c": 72, "b": 24, "e": 72, "d": 72}, False),
    ("abcd-ebad-ce", {"a": 96, "c": 24, "b": 84, "e": 96, "d": 84}, {"a": 72, "c": 24, "b": 72, "e": 72, "d": 72}, True),
    ("abcde-efbad-cf", {"a": 48, "c": 24, "b": 36, "e": 48, "d": 36, "f": 36}, {"a": 48, "c": 24, "b": 32, "e": 48, "d": 32, "f": 32}, False),
    ("abcde-ecbfa-fd", {"a": 48, "c": 36, "b": 36, "e": 48, "d": 24, "f": 48}, {"a": 48, "c": 32, "b": 32, "e": 48, "d": 24, "f": 48}, False),
    ("abcde-efcad-bf", {"a": 48, "c": 36, "b": 24, "e": 48, "d": 36, "f": 36}, {"a": 48, "c": 32, "b": 24, "e": 48, "d": 32, "f": 32}, False),
    ("abcd-ea-ebcd", {"a": 96, "c": 84, "b": 84, "e": 96, "d": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72}, True),
    ("abcd-eb-aecd", {"a": 96, "c": 84, "b": 84, "e": 96, "d": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72}, True),
    ("abcd-ec-abed", {"a": 96, "c": 84, "b": 84, "e": 96, "d": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72}, True),
    ("ab-ac-cb", {"a": 7248, "c": 7248, "b": 7240}, {"a": 5136, "c": 5136, "b": 5120}, True),
    ("ab-acd-dbc", {"a": 384, "c": 376, "b": 376, "d": 384}, {"a": 312, "c": 296, "b": 296, "d": 312}, True),
    ("ab-cad-dcb", {"a": 384, "c": 384, "b": 376, "d": 384}, {"a": 312, "c": 312, "b": 296, "d": 312}, False),
    ("abc-acd-db", {"a": 384, "c": 376, "b": 376, "d": 384}, {"a": 312, "c": 296, "b": 296, "d": 312}, True),
    ("abc-ad-bdc", {"a": 384, "c": 376, "b": 384, "d": 376}, {"a": 312, "c": 296, "b": 312, "d": 296}, True),
    ("abc-adc-bd", {"a": 384, "c": 376, "b": 384, "d": 376}, {"a": 312, "c": 296, "b": 312, "d": 296}, True),
    ("abc-adc-db", {"a": 384, "c": 376, "b": 376, "d": 384}, {"a": 312, "c": 296, "b": 296, "d": 312}, True),
    ("abc-adec-ebd", {"a": 96, "c": 84, "b": 84, "e": 96, "d": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72}, True),
    ("abcd-aebf-dfce", {"a": 96, "c": 84, "b": 84, "e": 84, "d": 96, "f": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aebf-fdec", {"a": 96, "c": 84, "b": 84, "e": 84, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aecf-bfde", {"a": 96, "c": 84, "b": 96, "e": 84, "d": 84, "f": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aecf-fbed", {"a": 96, "c": 84, "b": 84, "e": 84, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aedf-bfce", {"a": 96, "c": 84, "b": 96, "e": 84, "d": 84, "f": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aedf-fbec", {"a": 96, "c": 84, "b": 84, "e": 84, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aefb-fdce", {"a": 96, "c": 84, "b": 84, "e": 84, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-aefc-fbed", {"a": 96, "c": 84, "b": 84, "e": 84, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-eafb-fdec", {"a": 96, "c": 84, "b": 84, "e": 96, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, False),
    ("abcd-eafc-bfde", {"a": 96, "c": 84, "b": 96, "e": 96, "d": 84, "f": 84}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, True),
    ("abcd-eafd-fbec", {"a": 96, "c": 84, "b": 84, "e": 96, "d": 84, "f": 96}, {"a": 72, "c": 72, "b": 72, "e": 72, "d": 72, "f": 72}, False),
    ("abcdef-dega-gfbc", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, False),
    ("abcdef-degb-gfac", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-degc-gfab", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-dfga-gebc", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, False),
    ("abcdef-dfgb-geac", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-dfgc-geab", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-efga-gdbc", {"a": 24, "c": 20, "b": 20, "e": 24, "d": 20, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 24, "d": 16, "g": 24, "f": 16}, False),
    ("abcdef-efgb-gdac", {"a": 24, "c": 20, "b": 20, "e": 24, "d": 20, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 24, "d": 16, "g": 24, "f": 16}, True),
    ("abcdef-efgc-gdab", {"a": 24, "c": 20, "b": 20, "e": 24, "d": 20, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 24, "d": 16, "g": 24, "f": 16}, True),
    ("abcdef-gdab-efgc", {"a": 24, "c": 20, "b": 20, "e": 24, "d": 20, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 24, "d": 16, "g": 24, "f": 16}, True),
    ("abcdef-gdac-efgb", {"a": 24, "c": 20, "b": 20, "e": 24, "d": 20, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 24, "d": 16, "g": 24, "f": 16}, True),
    ("abcdef-gdbc-efga", {"a": 24, "c": 20, "b": 20, "e": 24, "d": 20, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 24, "d": 16, "g": 24, "f": 16}, False),
    ("abcdef-geab-dfgc", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-geac-dfgb", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-gebc-dfga", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, False),
    ("abcdef-gfab-degc", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-gfac-degb", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, True),
    ("abcdef-gfbc-dega", {"a": 24, "c": 20, "b": 20, "e": 20, "d": 24, "g": 24, "f": 20}, {"a": 24, "c": 16, "b": 16, "e": 16, "d": 24, "g": 24, "f": 16}, False),
]


def appendix_workloads(dtype: str = "f32") -> List[Workload]:
    """The 48 contractions as workloads at the extents of Table III (f32) or
    Table IV (f64)."""
    ws = []
    for i, (name, sp, dp, _) in enumerate(TABLE):
        c, a, b = name.split("-")
        ext = sp if dtype == "f32" else dp
        tag = f"appA{i + 1:02d}_{name}_{'fp32' if dtype == 'f32' else 'fp64'}"
        number = 2000 + i + (100 if dtype == "f64" else 0)
        ws.append(Workload(number, tag, dtype, ",".join(c), ",".join(a), ",".join(b), dict(ext)))
    return ws


def log_applicable() -> Dict[str, bool]:
    """Per contraction, whether the paper reports a LoG result."""
    return {name: ok for name, _, _, ok in TABLE}

