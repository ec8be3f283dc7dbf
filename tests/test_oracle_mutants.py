"""Plant plausible mistakes in copies of the oracle and check the pins catch each.

Every mutant is a textual edit of oracle/attn_ref.c compiled into a temporary
directory; the oracle itself is never modified. A mutant that passes every pin
would mean the pins cannot tell that mistake from the truth.
"""
import os

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "attn_ref.c")

MUTANTS = [
    ("scale dropped", "double s = p->scale * dot;", "double s = dot;"),
    ("softcap missing outer C", "s = p->softcap * tanh(s / p->softcap);", "s = tanh(s / p->softcap);"),
    ("softcap after ALiBi", "if (p->softcap > 0.0) s = p->softcap * tanh(s / p->softcap);\n    if (p->slopes) {\n        int64_t rel = i + (lk - lq) - j;\n        s -= p->slopes[h] * (double)(rel < 0 ? -rel : rel);\n    }",
     "if (p->slopes) {\n        int64_t rel = i + (lk - lq) - j;\n        s -= p->slopes[h] * (double)(rel < 0 ? -rel : rel);\n    }\n    if (p->softcap > 0.0) s = p->softcap * tanh(s / p->softcap);"),
    ("ALiBi sign", "s -= p->slopes[h]", "s += p->slopes[h]"),
    ("ALiBi signed distance", "(double)(rel < 0 ? -rel : rel)", "(double)rel"),
    ("ALiBi slope of kv head", "s -= p->slopes[h]", "s -= p->slopes[h / (p->hq / p->hkv)]"),
    ("causal strict", "if (p->mask_kind == 1) return j <= ii;", "if (p->mask_kind == 1) return j < ii;"),
    ("causal top-left", "int64_t ii = i + (lk - lq); /* query position", "int64_t ii = i; /* query position"),
    ("window left off by one", "ii - j > p->window_left", "ii - j >= p->window_left"),
    ("window right ignored", "if (p->window_right >= 0 && j - ii > p->window_right) return 0;", ""),
    ("GQA modulo map", "int32_t hk = h / group;", "int32_t hk = h % p->hkv;"),
    ("LSE without max", "lse[row] = mx + log(z);", "lse[row] = log(z);"),
    ("no normalisation", "double pj = exp(s[j] - mx) / z;", "double pj = exp(s[j] - mx);"),
    ("sum without max shift", "z += exp(s[j] - mx);", "z += exp(s[j]);"),
    ("V used as K", "score(p, qi, kbase + j * kstride", "score(p, qi, vbase + j * kstride"),
    ("varlen keys from sequence 0", "kbase = k + ((int64_t)p->cu_k[b] * p->hkv + hk) * p->d;",
     "kbase = k + ((int64_t)0 * p->hkv + hk) * p->d;"),
    ("varlen key length from queries", "lk = p->cu_k[b + 1] - p->cu_k[b];", "lk = lq;"),
    ("empty row LSE zero", "lse[row] = -INFINITY;", "lse[row] = 0.0;"),
    ("prefix inclusive of L_p", "if (j < p->prefix_len) return 1;", "if (j <= p->prefix_len) return 1;"),
    ("prefix without causal part", "return j <= ii;                  /* causal generation */",
     "return 0;"),
    ("relative position sign", "if (p->relpos) s += (double)(i + (lk - lq) - j);",
     "if (p->relpos) s += (double)(j - i - (lk - lq));"),
    ("relative position top-left", "if (p->relpos) s += (double)(i + (lk - lq) - j);",
     "if (p->relpos) s += (double)(i - j);"),
    # the relative-position line moved in front of the soft-cap (not duplicated)
    ("relative position before soft-cap",
     "    if (p->softcap > 0.0) s = p->softcap * tanh(s / p->softcap);\n"
     "    if (p->slopes) {\n"
     "        int64_t rel = i + (lk - lq) - j;\n"
     "        s -= p->slopes[h] * (double)(rel < 0 ? -rel : rel);\n"
     "    }\n"
     "    if (p->relpos) s += (double)(i + (lk - lq) - j);\n",
     "    if (p->relpos) s += (double)(i + (lk - lq) - j);\n"
     "    if (p->softcap > 0.0) s = p->softcap * tanh(s / p->softcap);\n"
     "    if (p->slopes) {\n"
     "        int64_t rel = i + (lk - lq) - j;\n"
     "        s -= p->slopes[h] * (double)(rel < 0 ? -rel : rel);\n"
     "    }\n"),
    # top-left alignment (query i at key position i instead of i + Lk - Lq),
    # one variant at a time; the window checks of the sliding window (first
    # occurrence) and of the global sliding window (second) are the same text
    ("ALiBi top-left", "int64_t rel = i + (lk - lq) - j;", "int64_t rel = i - j;"),
    ("window top-left",
     "if (p->window_left >= 0 && ii - j > p->window_left) return 0;\n"
     "        if (p->window_right >= 0 && j - ii > p->window_right) return 0;",
     "if (p->window_left >= 0 && i - j > p->window_left) return 0;\n"
     "        if (p->window_right >= 0 && j - i > p->window_right) return 0;", 0),
    ("global window band top-left",
     "if (p->window_left >= 0 && ii - j > p->window_left) return 0;\n"
     "        if (p->window_right >= 0 && j - ii > p->window_right) return 0;",
     "if (p->window_left >= 0 && i - j > p->window_left) return 0;\n"
     "        if (p->window_right >= 0 && j - i > p->window_right) return 0;", 1),
    ("global rows top-left", "if (in_global(p, ii) || in_global(p, j)) return 1;",
     "if (in_global(p, i) || in_global(p, j)) return 1;"),
    ("PrefixLM top-left", "return j <= ii;                  /* causal generation */",
     "return j <= i;"),
    ("share question top-left",
     "if (j > ii || ii < 0) return 0;\n        int32_t idi = p->token_ids[ii], idj = p->token_ids[j];",
     "if (j > i) return 0;\n        int32_t idi = p->token_ids[i], idj = p->token_ids[j];"),
    ("causal blockwise top-left",
     "if (ii >= p->query_start) return 1;          /* test query visibility   */\n"
     "        return p->token_ids[ii] == p->token_ids[j];",
     "if (i >= p->query_start) return 1;\n        return p->token_ids[i] == p->token_ids[j];"),
    ("causal blockwise causal part top-left",
     "if (j > ii || ii < 0) return 0;\n        if (ii >= p->query_start)",
     "if (j > i) return 0;\n        if (ii >= p->query_start)"),
    ("norm L from the query length", "double pj = a / (double)lk;", "double pj = a / (double)lq;"),
    ("norm without 1/L", "double pj = a / (double)lk;", "double pj = a;"),
    ("ReLU passes negatives", "a = s[j] > 0.0 ? s[j] : 0.0;", "a = s[j];"),
    ("Sigmoid sign", "a = 1.0 / (1.0 + exp(-s[j]));", "a = 1.0 / (1.0 + exp(s[j]));"),
    ("global rows not global", "if (in_global(p, ii) || in_global(p, j)) return 1;",
     "if (in_global(p, j)) return 1;"),
    ("global keys not global", "if (in_global(p, ii) || in_global(p, j)) return 1;",
     "if (in_global(p, ii)) return 1;"),
    ("response blind to prompt", "return idj < 0 || idj == idi;    /* response -> prompt + itself   */",
     "return idj == idi;"),
    ("test query starts one late", "if (ii >= p->query_start) return 1;          /* test query visibility   */",
     "if (ii > p->query_start) return 1;"),
    ("blockwise across documents", "return p->token_ids[ii] == p->token_ids[j];  /* demonstration isolation */",
     "return 1;"),
]


def _mutate(src, old, new, nth=None):
    """Replace every occurrence of `old`, or only the nth (0-based)."""
    if nth is None:
        return src.replace(old, new)
    at = -1
    for _ in range(nth + 1):
        at = src.index(old, at + 1)
    return src[:at] + new + src[at + len(old):]


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, mutant):
    name, old, new = mutant[:3]
    nth = mutant[3] if len(mutant) > 3 else None
    src = open(SRC).read()
    assert src.count(old) > (nth or 0), f"mutation site for '{name}' not found"
    mutated = _mutate(src, old, new, nth)
    assert mutated != src
    path = tmp_path / "attn_ref_mutant.c"
    path.write_text(mutated)
    so = oracle.build(str(path), str(tmp_path / "libmutant.so"))
    lib = oracle.load(so)
    failed = oracle_pins.failing_pins(lib)
    assert failed, f"no pin catches the mutant '{name}'"
