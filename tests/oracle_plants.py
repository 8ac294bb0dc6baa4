"""Planted mistakes in the oracle: every one must fail a CPU pin (not collected by pytest).

    python tests/oracle_plants.py [-j 6] [-k NAME]

Each plant is one plausible mistake (a dropped clause, a wrong sign, index, order or rounding)
written as an exact text replacement in one oracle file.  For every plant the script copies
``oracle/``, ``tests/`` and ``workloads/`` to a scratch directory, applies the replacement there
(never in the tree), runs the oracle pins (``tests/test_oracle_*.py``), and reports whether some
test failed.  Plants marked ``equivalent`` change no result by construction (the reason is given);
they are listed so that nobody counts them as unpinned.  Exit status 1 if a non-equivalent plant
passes every pin.
"""

from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, file, old text, new text, equivalent-because or None)
PLANTS = [
    # ---- ARC (oracle/arc.py): cases, REPLACE, adaptation, ghosts, victim window
    ("replace_no_tie", "oracle/arc.py", "(n1 > self.p or (x_in_b2 and n1 == self.p))", "(n1 > self.p)", None),
    ("replace_tie_any_ref", "oracle/arc.py", "(n1 > self.p or (x_in_b2 and n1 == self.p))", "(n1 >= self.p)", None),
    ("replace_ge", "oracle/arc.py", "prefer_t1 = n1 > 0 and (n1 > self.p or", "prefer_t1 = n1 > 0 and (n1 >= self.p or", None),
    ("case2_tie_clause", "oracle/arc.py", "evicted, evicted_from, phys = self._replace(False)\n            del self.B1[x]",
     "evicted, evicted_from, phys = self._replace(True)\n            del self.B1[x]", None),
    ("delta2_one", "oracle/arc.py", "d2 = 1.0 if len(self.B2) >= len(self.B1) else len(self.B1) / len(self.B2)", "d2 = 1.0", None),
    ("delta2_floor", "oracle/arc.py", "else len(self.B1) / len(self.B2)", "else float(len(self.B1) // len(self.B2))", None),
    ("delta2_inverse", "oracle/arc.py", "else len(self.B1) / len(self.B2)", "else len(self.B2) / len(self.B1)", None),
    ("delta1_inverse", "oracle/arc.py", "else len(self.B2) / len(self.B1)", "else len(self.B1) / len(self.B2)", None),
    ("delta1_strict", "oracle/arc.py", "d1 = 1.0 if len(self.B1) >= len(self.B2)", "d1 = 1.0 if len(self.B1) > len(self.B2)",
     "at |B1| = |B2| the ratio is 1 as well"),
    ("delta2_strict", "oracle/arc.py", "d2 = 1.0 if len(self.B2) >= len(self.B1)", "d2 = 1.0 if len(self.B2) > len(self.B1)",
     "at |B1| = |B2| the ratio is 1 as well"),
    ("p_no_cap", "oracle/arc.py", "self.p = min(self.p + d1, float(c))", "self.p = self.p + d1", None),
    ("p_no_floor", "oracle/arc.py", "self.p = max(self.p - d2, 0.0)", "self.p = self.p - d2", None),
    ("case2_replace_after_p", "oracle/arc.py",
     "self.p = min(self.p + d1, float(c))\n            evicted, evicted_from, phys = self._replace(False)",
     "evicted, evicted_from, phys = self._replace(False)\n            self.p = min(self.p + d1, float(c))", None),
    ("case3_replace_after_p", "oracle/arc.py",
     "self.p = max(self.p - d2, 0.0)\n            evicted, evicted_from, phys = self._replace(True)",
     "evicted, evicted_from, phys = self._replace(True)\n            self.p = max(self.p - d2, 0.0)", None),
    ("hit_stays_in_t1", "oracle/arc.py",
     "phys = self.T1.pop(x) if x in self.T1 else self.T2.pop(x)\n            self.T2[x] = phys",
     "if x in self.T1:\n                self.T1.move_to_end(x); phys = self.T1[x]\n            else:\n"
     "                phys = self.T2.pop(x); self.T2[x] = phys", None),
    ("b1_hit_to_t1", "oracle/arc.py", "del self.B1[x]\n            self.T2[x] = phys", "del self.B1[x]\n            self.T1[x] = phys", None),
    ("b2_hit_to_t2_lru", "oracle/arc.py", "del self.B2[x]\n            self.T2[x] = phys",
     "del self.B2[x]\n            self.T2[x] = phys\n            self.T2.move_to_end(x, last=False)", None),
    ("ghost_at_lru_end", "oracle/arc.py", "ghost[victim] = None", "ghost[victim] = None\n                ghost.move_to_end(victim, last=False)", None),
    ("iva_drops_b1_mru", "oracle/arc.py", "dropped = next(iter(self.B1))", "dropped = next(reversed(self.B1))", None),
    ("iva_t1_le_c", "oracle/arc.py", "if len(self.T1) < c:", "if len(self.T1) <= c:", None),
    ("iva_t1del_keeps_ghost", "oracle/arc.py", "dropped, dropped_from = victim, FROM_T1",
     "dropped, dropped_from = victim, FROM_T1\n                    self.B1[victim] = None", None),
    ("iva_t1del_mru", "oracle/arc.py",
     "victim = self._lru_unpinned(self.T1)\n                    if victim is None:\n"
     "                        raise RuntimeError(\"IV-A: every T1 page is pinned\")",
     "victim = next(reversed(self.T1))", None),
    ("ivb_total_gt_c", "oracle/arc.py", "if total >= c:", "if total > c:", None),
    ("ivb_2c_drops_b1", "oracle/arc.py", "dropped = next(iter(self.B2))\n                        del self.B2[dropped]",
     "dropped = next(iter(self.B1)) if self.B1 else next(iter(self.B2))\n"
     "                        (self.B1 if self.B1 else self.B2).pop(dropped)", None),
    ("ivb_2c_drops_b2_mru", "oracle/arc.py", "dropped = next(iter(self.B2))", "dropped = next(reversed(self.B2))", None),
    ("window_ties_to_newer", "oracle/arc.py", "if best is None or depth.get(key, 0) > depth.get(best, 0):",
     "if best is None or depth.get(key, 0) >= depth.get(best, 0):", None),
    ("window_one_too_wide", "oracle/arc.py", "        seen += 1\n        if seen == window:",
     "        seen += 1\n        if seen == window + 1:", None),
    # ---- LRU (oracle/lru.py)
    ("lru_hit_not_moved", "oracle/lru.py", "            self.L.move_to_end(x)\n            ev = Event", "            ev = Event", None),
    ("lru_evicts_mru", "oracle/lru.py", "victim = window_victim(self.L, self.pinned, self.depth, self.window)",
     "victim = next(reversed(self.L))", None),
    ("lru_capacity_off_by_one", "oracle/lru.py", "if len(self.L) == self.c:", "if len(self.L) == self.c - 1:", None),
    # ---- attention (oracle/attention.py)
    ("att_mask_strict", "oracle/attention.py", "visible = np.arange(L)[None, :] <= positions[:, None]",
     "visible = np.arange(L)[None, :] < positions[:, None]", None),
    ("att_no_max_shift", "oracle/attention.py", "w = np.exp(s - m)", "w = np.exp(s)", None),
    ("att_gqa_modulo", "oracle/attention.py", "kh = h // g", "kh = h % hkv", None),
    ("att_position_off_by_one", "oracle/attention.py", "pos = prefix_len + rs", "pos = prefix_len + rs - 1", None),
    ("att_no_scale", "oracle/attention.py", "s = scale * (q @ k.T)", "s = (q @ k.T)", None),
    # ---- KV pool (oracle/kvpool.py)
    ("pool_gather_offset", "oracle/kvpool.py", "off = j % BLOCK_TOKENS\n    k = k_pool", "off = (j + 1) % BLOCK_TOKENS\n    k = k_pool", None),
    ("pool_v_token_major", "oracle/kvpool.py", "v_pool[blk, :, :, off] = v_new", "v_pool[blk, :, off, :] = v_new", None),
    # ---- planner (oracle/planner.py)
    ("plan_whole_prompt_hit", "oracle/planner.py", "            if BLOCK_TOKENS * k == n_tok:\n                k -= 1", "            pass", None),
    ("plan_head_first", "oracle/planner.py",
     "order = range(n_full - 1, -1, -1) if self.ref_order == \"tail_first\" else range(n_full)", "order = range(n_full)", None),
    ("plan_prefix_unpinned", "oracle/planner.py", "            for i in range(k):\n                cache.pin(hashes[i])", "            pass", None),
    ("plan_slot_offset", "oracle/planner.py",
     "plan.slot_mapping.append(row[j // BLOCK_TOKENS] * BLOCK_TOKENS + j % BLOCK_TOKENS)",
     "plan.slot_mapping.append(row[j // BLOCK_TOKENS] * BLOCK_TOKENS + (j + 1) % BLOCK_TOKENS)", None),
    ("plan_scratch_lifo", "oracle/planner.py", "blk = self.scratch.popleft()", "blk = self.scratch.pop()", None),
    ("plan_scratch_back_at_head", "oracle/planner.py", "self.scratch.extend(self.batch_scratch)",
     "self.scratch.extendleft(self.batch_scratch)", None),
    ("plan_b2_hit_not_born", "oracle/planner.py", "if ev.case not in (CASE_I, LRU_HIT):      # a miss or a ghost hit",
     "if ev.case not in (CASE_I, LRU_HIT) and ev.case != 2:", None),
    ("plan_b1_hit_not_born", "oracle/planner.py", "if ev.case not in (CASE_I, LRU_HIT):      # a miss or a ghost hit",
     "if ev.case not in (CASE_I, LRU_HIT) and ev.case != 1:", None),
    ("batch_budget_strict", "oracle/planner.py", "if blocks + nf > capacity or tails + tl > scratch_blocks:",
     "if blocks + nf >= capacity or tails + tl > scratch_blocks:", None),
    # ---- block hash (oracle/blockhash.py)
    ("fnv_multiply_then_xor", "oracle/blockhash.py", "        h ^= b\n        h = (h * FNV_PRIME) & MASK64",
     "        h = (h * FNV_PRIME) & MASK64\n        h ^= b", None),
    ("hash_parent_big_endian", "oracle/blockhash.py", 'out = int(parent & MASK64).to_bytes(8, "little")',
     'out = int(parent & MASK64).to_bytes(8, "big")', None),
    ("hash_root_ignored", "oracle/blockhash.py", "h = root & MASK64\n    for i in range(n_full):",
     "h = FNV_OFFSET\n    for i in range(n_full):", None),
    ("hash_many_parent_of_finished", "oracle/blockhash.py", "parent = np.where(live, h, parent)", "parent = h",
     "a finished sequence is never live again, so its parent is never read"),
    # ---- Q/K/V producer (oracle/qkv.py)
    ("bf16_truncates", "oracle/qkv.py", "r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16", "r = u >> 16", None),
    ("rope_sign", "oracle/qkv.py", "return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)",
     "return np.concatenate([lo * c + hi * s, hi * c - lo * s], axis=-1)", None),
    ("rope_frequency", "oracle/qkv.py", "f = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d)",
     "f = theta ** (-1.0 * np.arange(half, dtype=np.float64) / d)", None),
    ("rope_reads_unrounded_y", "oracle/qkv.py", "y = bf16_to_f64(f64_to_bf16_bits(project(x_bits, w_bits)))",
     "y = project(x_bits, w_bits)", None),
    ("v_rotated", "oracle/qkv.py", "v = y[:, nq + nk:nq + 2 * nk].reshape(t, num_kv_heads, head_dim)",
     "v = rope(y[:, nq + nk:nq + 2 * nk].reshape(t, num_kv_heads, head_dim), positions, theta)", None),
    ("positions_from_zero", "oracle/qkv.py", "out.append(np.arange(int(seq_lens[r]) - s, int(seq_lens[r])))",
     "out.append(np.arange(0, s))", None),
]


def run_one(plant):
    name, rel, old, new, _ = plant
    with tempfile.TemporaryDirectory(prefix=f"plant_{name}_") as d:
        for sub in ("oracle", "tests", "workloads"):
            shutil.copytree(os.path.join(ROOT, sub), os.path.join(d, sub),
                            ignore=shutil.ignore_patterns("__pycache__"))
        shutil.copy(os.path.join(ROOT, "pytest.ini"), d)
        path = os.path.join(d, rel)
        src = open(path).read()
        if src.count(old) != 1:
            return name, "stale", f"text to replace found {src.count(old)} times in {rel}"
        open(path, "w").write(src.replace(old, new))
        tests = sorted(os.path.join("tests", f) for f in os.listdir(os.path.join(d, "tests"))
                       if f.startswith("test_oracle_") and f.endswith(".py"))
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *tests],
                           cwd=d, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        failed = [l.split("::")[-1].split(" ")[0] for l in r.stdout.splitlines() if l.startswith("FAILED")]
        return name, "caught" if r.returncode != 0 else "passed", ", ".join(failed)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=6)
    ap.add_argument("-k", default="")
    a = ap.parse_args()
    plants = [p for p in PLANTS if a.k in p[0]]
    with ThreadPoolExecutor(a.j) as ex:
        results = list(ex.map(run_one, plants))
    bad = 0
    for (name, status, detail), plant in zip(results, plants):
        equiv = plant[4]
        tag = f"equivalent ({equiv})" if equiv else status
        if not equiv and status != "caught":
            bad += 1
        print(f"{name:32s} {tag:12s} {detail}")
    n_eq = sum(1 for p in plants if p[4])
    print(f"{len(plants)} plants, {n_eq} equivalent, {bad} non-equivalent plants not caught")
    sys.exit(1 if bad else 0)


if __name__ == "__main__":
    main()
