"""Pins of the oracle's TIDE pass on hand-worked traces (tests/tide_cases.py):
a promote-only move into free SRAM, a swap that frees SRAM followed by a
promote-only move that brings back the session demoted earlier, a pass that
ends because the budget runs out mid-loop, and a pass that ends at its first
illegal move although a later candidate would be legal.  Exact decision
lists, budgets, moved bytes and prefetch hits.  No GPU."""
import numpy as np
import pytest

import oracle
import tide_cases

H0 = (np.zeros(51, np.uint32), np.ones(51, np.uint32))


@pytest.mark.parametrize("name", sorted(tide_cases.CASES))
def test_tide_worked_example(name):
    tr, p, want_log, want, budgets = tide_cases.CASES[name]()
    rc, cnt, log, st, _ = oracle.run(tr, p[0], H0[0], H0[1], log_cap=1000, states=True)
    assert rc == 0
    got = [(int(r["ev"]), int(r["op"]), int(r["a"]), int(r["b"])) for r in log]
    assert got == want_log
    for k, v in want.items():
        assert cnt[k] == v, (k, cnt[k], v)
    for e, (budget, moved) in budgets.items():
        assert st[e]["tide_ran"] == 1
        assert (int(st[e]["tide_budget"]), int(st[e]["tide_moved"])) == (budget, moved), e
    assert cnt["hit_sram"] + cnt["hit_hbm"] + cnt["miss"] == cnt["requests"] == len(
        [1 for r in range(tr.n_events) if tr.kind[r] == 0])


# Plausible mistakes in the TIDE pass, each planted in a temporary copy of the
# oracle's source: (name, text replaced, replacement).
SKIP_TO_FITTING = '''
static uint32_t argmin_movable(const sim_t* m, uint64_t left) {
  uint32_t best = NONE_ID;
  uint64_t bk = 0;
  for (uint32_t i = 0; i < m->n_sess; i++) {
    if (!evictable(&m->s[i]) || m->s[i].tier != T_HBM) continue;
    uint64_t sz = size_of(m, i);
    if (m->used[T_SRAM] + sz > m->p->cap_sram_B || sz > left) continue;
    uint64_t k = key_of(m, i);
    if (best == NONE_ID || k < bk) { best = i; bk = k; }
  }
  return best == NONE_ID ? argmin_key(m, T_HBM) : best;
}

/* Algorithm 1, tiering branch'''
MUTANTS = [
    ("promote ignores the budget",
     "if (m->used[T_SRAM] + sp <= p->cap_sram_B && sp <= left) {",
     "if (m->used[T_SRAM] + sp <= p->cap_sram_B) {"),
    ("no promote-only move",
     "if (m->used[T_SRAM] + sp <= p->cap_sram_B && sp <= left) {",
     "if (0) {"),
    ("swap tried before the promote-only move",
     "uint32_t did = argmax_key(m, T_SRAM);\n    if (did == NONE_ID) break;",
     "uint32_t did = argmax_key(m, T_SRAM);\n    if (did == NONE_ID) break;\n"
     "    if (0) {}"),
    ("swap on equal keys", "int legal = kp < kd &&", "int legal = kp <= kd &&"),
    ("swap ignores SRAM capacity", "m->used[T_SRAM] - sd + sp <= p->cap_sram_B &&", ""),
    ("swap ignores the budget", "sp <= left && sd <= left - sp &&", ""),
    ("swap-in not marked as prefetched",
     "m->s[pid].prefetched = 1;\n    m->s[did].tier = T_HBM;",
     "m->s[did].tier = T_HBM;"),
    ("an illegal candidate is skipped, not the end of the pass",
     "uint32_t pid = argmin_key(m, T_HBM);", "uint32_t pid = argmin_movable(m, left);"),
]


SWAP_FIRST = """    uint64_t sp = size_of(m, pid);
    uint32_t did = argmax_key(m, T_SRAM);
    if (did != NONE_ID) {
      uint64_t kd = key_of(m, did);
      uint64_t sd = size_of(m, did);
      if (kp < kd && sp <= left && sd <= left - sp &&
          m->used[T_SRAM] - sd + sp <= p->cap_sram_B && m->used[T_HBM] - sp + sd <= p->cap_hbm_B) {
        m->used[T_SRAM] = m->used[T_SRAM] - sd + sp;
        m->used[T_HBM] = m->used[T_HBM] - sp + sd;
        m->s[pid].tier = T_SRAM;
        m->s[pid].prefetched = 1;
        m->s[did].tier = T_HBM;
        left -= sp + sd;
        moved += sp + sd;
        emit(m, OP_SWAP, pid, did);
        m->c->swap++;
        continue;
      }
    }
    if (m->used[T_SRAM] + sp <= p->cap_sram_B && sp <= left) {
      m->used[T_HBM] -= sp;
      m->used[T_SRAM] += sp;
      m->s[pid].tier = T_SRAM;
      m->s[pid].prefetched = 1;
      left -= sp;
      moved += sp;
      emit(m, OP_PROMOTE, pid, NONE_ID);
      m->c->promote++;
      continue;
    }
    break;
  }
  m->keysrc = src;"""


def _swap_first(src):
    # the swap with the HBM minimum is tried first; a promote-only move only
    # when no swap is legal
    a = src.index("    uint64_t sp = size_of(m, pid);\n")
    b = src.index("  }\n  m->keysrc = src;", a)
    return src[:a] + SWAP_FIRST + src[b + len("  }\n  m->keysrc = src;"):]


@pytest.mark.parametrize("k", range(len(MUTANTS)))
def test_each_planted_tide_mistake_fails_a_pin(tmp_path, k):
    name, old, new = MUTANTS[k]
    src = oracle.source_text()
    assert src.count(old) == 1, name
    if name.startswith("swap tried before"):
        src = _swap_first(src)
    else:
        src = src.replace(old, new)
    if "argmin_movable" in new:
        src = src.replace("\n/* Algorithm 1, tiering branch", SKIP_TO_FITTING, 1)
    lib = oracle.load_library(oracle.compile_source(src, str(tmp_path / "mutant.so")))
    caught = []
    for case, build in sorted(tide_cases.CASES.items()):
        tr, p, want_log, want, budgets = build()
        rc, cnt, log, st, _ = oracle.run(tr, p[0], H0[0], H0[1], log_cap=1000, states=True,
                                         library=lib)
        got = [(int(r["ev"]), int(r["op"]), int(r["a"]), int(r["b"])) for r in log]
        if rc != 0 or got != want_log or any(cnt[f] != v for f, v in want.items()) or any(
                (int(st[e]["tide_budget"]), int(st[e]["tide_moved"])) != bm
                for e, bm in budgets.items()):
            caught.append(case)
    assert caught, "planted mistake not caught: " + name
