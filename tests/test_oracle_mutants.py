"""Plant plausible mistakes in copies of oracle.c and require the pins to catch
each one (CPU only).  Nothing here touches the real oracle build."""
import os
import shutil
import tempfile

import pytest

import oracle
from oracle import build as obuild
from oracle_pins import ALL_PINS

SRC = os.path.join(os.path.dirname(obuild.__file__), "oracle.c")

# (name, text in oracle.c, replacement)
MUTANTS = [
    ("scale dropped", "score[j] = a->scale * dot;", "score[j] = dot;"),
    ("window one short", "j >= p - a->window + 1", "j >= p - a->window + 2"),
    ("window one long", "j >= p - a->window + 1", "j >= p - a->window"),
    ("causal excludes own token", "if (j > p) return 0;", "if (j >= p) return 0;"),
    ("no causal mask", "if (j > p) return 0;", "if (j > p + 1000000) return 0;"),
    ("top-left alignment", "int p = S - a->q_len + i;", "int p = i;"),
    ("sinks one too many", "return j < a->n_sink ||", "return j <= a->n_sink ||"),
    ("GQA heads interleaved", "int hk = h / G;", "int hk = h % a->Hkv;"),
    ("K and V swapped in scores", "load_elem(a->k, a->dtype, k_off + c);",
     "load_elem(a->v, a->dtype, k_off + c);"),
    ("lse without max", "m + log(Z) : -INFINITY", "log(Z) : -INFINITY"),
    ("lse in log2", "m + log(Z) : -INFINITY", "m + log2(Z) : -INFINITY"),
    ("row order transposed", "int h = (int)(row % a->Hq);\n    int i = (int)((row / a->Hq) % a->q_len);",
     "int i = (int)(row % a->q_len);\n    int h = (int)((row / a->q_len) % a->Hq);"),
    ("page slot wrong", "tok = j % a->page_size;", "tok = (j + 1) % a->page_size;"),
    ("bf16 widened wrongly", "[idx]) << 16;", "[idx]) << 15;"),
    ("merge without max shift", "total += exp(l - mx);", "total += exp(l);"),
    ("merge weight unnormalised", "double w = exp(l - lse_r);", "double w = exp(l - mx);"),
    ("indexed: speculated tokens not visible", "return j >= S - a->q_len || member[j];",
     "return member[j];"),
    ("indexed: list entries past idx_len used", "int n = a->idx_len[b] < a->idx_stride ? a->idx_len[b] : a->idx_stride;",
     "int n = a->idx_stride;"),
    ("indexed: list ignored (full cache)", "if (a->mode == ORACLE_VERIFY) return 1;",
     "if (a->mode != ORACLE_DRAFT) return 1;"),
    ("snapkv: pooling divisor off", "out[j] = s / pool;", "out[j] = s / (pool - 1);"),
    ("snapkv: pooling window shifted", "for (int t = j - pool / 2; t <= j + pool / 2; ++t)",
     "for (int t = j - pool / 2 + 1; t <= j + pool / 2 + 1; ++t)"),
    ("snapkv: window queries not causal", "for (int j = 0; j <= p && j < S; ++j)",
     "for (int j = 0; j < S; ++j)"),
    ("snapkv: ties to the larger position", "return i < j ? -1 : (i > j);\n}\nstatic int asc_cmp",
     "return i > j ? -1 : (i < j);\n}\nstatic int asc_cmp"),
    ("snapkv: observation window dropped", "for (int j = n; j < S; ++j) out[c++] = j;",
     "for (int j = S; j < S; ++j) out[c++] = j;"),
    ("merge keeps empty parts", "if (l == -INFINITY) continue;\n      double w",
     "if (0) continue;\n      double w"),
]


@pytest.fixture(scope="module")
def tmpdir_mod():
    d = tempfile.mkdtemp(prefix="oracle_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, old, new, tmpdir_mod):
    text = open(SRC).read()
    assert text.count(old) >= 1, f"mutation anchor not found: {old!r}"
    mutated = text.replace(old, new)
    tag = "".join(ch if ch.isalnum() else "_" for ch in name)
    src = os.path.join(tmpdir_mod, f"{tag}.c")
    with open(src, "w") as f:
        f.write(mutated)
    lib = oracle.open_library(obuild.build(src=src, out=os.path.join(tmpdir_mod, f"{tag}.so")))
    caught = []
    for pin in ALL_PINS:
        try:
            pin(lib=lib)
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake '{name}'"


# Planted mistakes in copies of oracle/sdstep.py: (name, text, replacement)
SDSTEP_SRC = os.path.join(os.path.dirname(obuild.__file__), "sdstep.py")
SDSTEP_MUTANTS = [
    ("accept: last draft never accepted", "while a < L - 1 and", "while a < L - 2 and"),
    ("accept: bonus from the next input", "tokens[b, a] = target[b, a]",
     "tokens[b, a] = target[b, min(a + 1, L - 1)]"),
    ("accept: ties to the last index", "return np.argmax(x, axis=-1).astype(np.int64)",
     "return (x.shape[-1] - 1 - np.argmax(x[..., ::-1], axis=-1)).astype(np.int64)"),
    ("accept: NaN wins", "x = np.where(np.isnan(x), -np.inf, x)", "x = x"),
    ("accept: bf16 widened wrongly", "astype(np.uint32) << 16", "astype(np.uint32) << 15"),
    ("eq1: exponent gamma", "alpha ** (gamma + 1)", "alpha ** gamma"),
    ("append: one slot late", "int(pos0[b]) + i,", "int(pos0[b]) + i + 1,"),
    ("append: page slot wrong", "return int(page_table[b, j // page_size]), j % page_size",
     "return int(page_table[b, j // page_size]), (j + 1) % page_size"),
    ("commit: bonus input not kept", "np.asarray(accepted, np.int64) + 1",
     "np.asarray(accepted, np.int64)"),
    ("ring: last kept position dropped", "range(C, C + int(accepted[b]) + 1)",
     "range(C, C + int(accepted[b]))"),
    ("ring: slot shifted", "idx[b, :, ring_start + j % ring_len] = j",
     "idx[b, :, ring_start + (j + 1) % ring_len] = j"),
    ("streaming: window one short", "range(max(n_sink, C - window), C)",
     "range(max(n_sink, C - window + 1), C)"),
    ("streaming: sinks dropped", "for j in range(min(n_sink, C)):", "for j in range(0):"),
    ("gather: the next head's row", "out[dblk, dtok, h] = src[sblk, stok, h]",
     "out[dblk, dtok, h] = src[sblk, stok, (h + 1) % Hkv]"),
    ("gather: unusable entries copied", "if 0 <= p < int(src_lens[b]):", "if 0 <= p < src.shape[1]:"),
    ("gather: destination row shifted", "dblk, dtok = cache_slot(b, j, dst_page_size",
     "dblk, dtok = cache_slot(b, j + 1, dst_page_size"),
    ("gather: source position off by one", "sblk, stok = cache_slot(b, p, src_page_size",
     "sblk, stok = cache_slot(b, p + 1, src_page_size"),
    ("gather: idx_len not clamped", "n = np.clip(np.asarray(idx_len, np.int64), 0, stride)",
     "n = np.asarray(idx_len, np.int64)"),
]


@pytest.mark.parametrize("name,old,new", SDSTEP_MUTANTS, ids=[m[0] for m in SDSTEP_MUTANTS])
def test_sdstep_mutant_is_caught(name, old, new):
    import importlib.util

    from sdstep_pins import ALL_SDSTEP_PINS

    text = open(SDSTEP_SRC).read()
    assert text.count(old) == 1, f"mutation anchor not found once: {old!r}"
    spec = importlib.util.spec_from_loader("sdstep_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(text.replace(old, new), "sdstep_mutant.py", "exec"), mod.__dict__)
    caught = []
    for pin in ALL_SDSTEP_PINS:
        try:
            pin(mod=mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake '{name}'"


# Planted mistakes in copies of oracle/costmodel.py.
COSTMODEL_SRC = os.path.join(os.path.dirname(obuild.__file__), "costmodel.py")
COSTMODEL_MUTANTS = [
    ("eq1: exponent gamma", "alpha ** (gamma + 1)", "alpha ** gamma"),
    ("eq1: alpha = 1 limit gamma", "return float(gamma + 1)", "return float(gamma)"),
    ("step: drafts not multiplied by gamma", "return gamma * draft_time(", "return 1 * draft_time("),
    ("eq3: selection ignored", "return t_draft + t_select", "return t_draft"),
    ("eq2: not divided by Omega", "expected_tokens(gamma, alpha) * t_target)", "1.0 * t_target)"),
    ("eq4: ties to the larger gamma", "if best is None or r < best[1]:", "if best is None or r <= best[1]:"),
    ("eq4: gamma off by one", "enumerate(t_verify_by_gamma, start=1)", "enumerate(t_verify_by_gamma, start=0)"),
    ("inverse: bisection reversed", "if expected_tokens(gamma, mid) < omega:", "if expected_tokens(gamma, mid) > omega:"),
]


@pytest.mark.parametrize("name,old,new", COSTMODEL_MUTANTS, ids=[m[0] for m in COSTMODEL_MUTANTS])
def test_costmodel_mutant_is_caught(name, old, new):
    import importlib.util

    from costmodel_pins import ALL_COSTMODEL_PINS

    text = open(COSTMODEL_SRC).read()
    assert text.count(old) == 1, f"mutation anchor not found once: {old!r}"
    spec = importlib.util.spec_from_loader("costmodel_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(text.replace(old, new), "costmodel_mutant.py", "exec"), mod.__dict__)
    caught = []
    for pin in ALL_COSTMODEL_PINS:
        try:
            pin(mod=mod)
        except (AssertionError, ValueError, ZeroDivisionError, TypeError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake '{name}'"
