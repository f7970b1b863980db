"""Plants plausible mistakes in copies of the oracle (on the CPU) and checks
that each one fails at least one pin, so the pins would catch them."""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")
HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

# (label, exact text in oracle.c, replacement)
MUTANTS = [
    ("tie-break reversed", "if (x->eid != y->eid) return x->eid < y->eid ? -1 : 1;",
     "if (x->eid != y->eid) return x->eid < y->eid ? 1 : -1;"),
    ("hop and etype swapped in the counter", "(uint32_t)hop,\n                     (uint32_t)etype}",
     "(uint32_t)etype,\n                     (uint32_t)hop}"),
    ("wrong output word", "uint32_t k = out[eid & 3];", "uint32_t k = out[(eid + 1) & 3];"),
    ("key truncation ignored", "if (key_bits < 32) k >>= (32 - key_bits);", ""),
    ("no round-key bump", "k0 += PHILOX_W0;", "k0 += 0;"),
    ("high half where the low half goes", "uint32_t y1 = lo1;", "uint32_t y1 = hi1;"),
    ("sigma high word dropped", "uint32_t key[2] = {(uint32_t)sigma, (uint32_t)(sigma >> 32)};",
     "uint32_t key[2] = {(uint32_t)sigma, 0u};"),
    ("take-all threshold off by one", "if (fanout < 0 || deg <= fanout) {",
     "if (fanout < 0 || deg <= fanout + 1) {"),
    ("largest keys kept", "for (int64_t j = 0; j < fanout; ++j) out_eids[j] = all[j].eid;",
     "for (int64_t j = 0; j < fanout; ++j) out_eids[j] = all[deg - 1 - j].eid;"),
    ("kept edges left in key order", "qsort(out_eids, (size_t)fanout, sizeof(int64_t), cmp_i64);", ""),
    ("hop index shifted in sampling",
     "int st = chosen ? select_pair(sigma, h, e, lo, hi, k, key_bits, excl[e].eids,",
     "int st = chosen ? select_pair(sigma, h + 1, e, lo, hi, k, key_bits, excl[e].eids,"),
    ("frontier not removed from new vertices",
     "if (find_gid_pos(ftab[t], fn[t], srcs[j]) >= 0) continue;", ""),
    ("new vertices left unsorted",
     "qsort(srcs, (size_t)m, sizeof(int64_t), cmp_i64);\n      /* unique",
     "/* unsorted */\n      /* unique"),
    ("new vertices numbered from 0", "if (pos < 0) pos = fn[s] + find_sorted(",
     "if (pos < 0) pos = find_sorted("),
    ("destination local ID off by one", "r->dst_local = (int32_t)i;",
     "r->dst_local = (int32_t)(i + 1);"),
    ("repeated seeds accepted", "if (i > 0 && tmp[i] == tmp[i - 1]) bad = 1;", ""),
    ("gather reads the mirrored row", "(const char *)feat + ids[i] * row_bytes",
     "(const char *)feat + ids[n - 1 - i] * row_bytes"),
    # edge-seeded mini-batches
    ("excluded edges still sampled",
     "if (nx == 0 || find_sorted(xs, nx, j) < 0) out_eids[deg++] = j;", "out_eids[deg++] = j;"),
    ("reverse edges not excluded",
     "excl[e].eids[m++] = batch->rev_eid[f][batch->eids[f][i]];", "(void)f;"),
    ("edge destination one slot late", "if (indptr[m] <= eid)", "if (indptr[m] < eid)"),
    ("negative from the wrong word",
     "uint64_t u = (uint64_t)out[0] | ((uint64_t)out[1] << 32);",
     "uint64_t u = (uint64_t)out[0] | ((uint64_t)out[2] << 32);"),
    ("negatives share the sampling counters", "0x80000000u | (uint32_t)k,", "(uint32_t)k,"),
    ("seeds not deduplicated", "if (a[i] != a[u - 1]) a[u++] = a[i];", "a[u++] = a[i];"),
    ("negative destinations left out of the seeds",
     "for (int64_t i = 0; i < n * Q; ++i) all[m++] = neg[e][i];", ""),
    ("pair source looked up among the destination type's seeds",
     "b->pos_src[e][i] = (int32_t)find_sorted(b->seed_gid[s], b->seed_n[s], src[e][i]);",
     "b->pos_src[e][i] = (int32_t)find_sorted(b->seed_gid[d], b->seed_n[d], src[e][i]);"),
    ("reverse edge not checked against the target",
     "if (etypes[r].indices[rj] != v || rv != et->indices[j]) return ORACLE_EINVAL;", ""),
    # layer-wise (LADIES) mini-batches
    ("importance from deg, not deg squared",
     "const unsigned __int128 d2 = (unsigned __int128)(uint64_t)deg * (uint64_t)deg;",
     "const unsigned __int128 d2 = (unsigned __int128)(uint64_t)deg;"),
    ("frontier left among the candidates", "if (in_f[s][u]) continue;", "(void)0;"),
    ("layer draws in the negatives' counter domain", "0x40000000u | (uint32_t)hop",
     "0x80000000u | (uint32_t)hop"),
    ("draw lands one candidate early", "if (pre[mid] <= r)", "if (pre[mid] < r)"),
    ("layer block keeps every in-edge", "if (pos < 0) continue;", "(void)0;"),
    ("every-candidate layer size ignored", "for (int64_t i = 0; i < nc; ++i) drawn[i] = 1;",
     "for (int64_t i = 0; i < nc; ++i) drawn[i] = 0;"),
    ("importance not cleared between hops", "        wt[t][cand[i]] = 0;\n", ""),
]


def fast_pins(lib):
    rng = np.random.default_rng(99)
    fails = []
    fails += pins.pin_philox(lib, rng, n=20)
    fails += pins.pin_edge_key(lib, rng, n=40)
    fails += pins.pin_select(lib, rng, n=60)
    fails += pins.pin_special_fanouts(lib, rng)
    fails += pins.pin_blocks(lib, rng, n=15)
    fails += pins.pin_gather(lib, rng, n=8)
    fails += pins.pin_errors(lib)
    fails += pins.pin_edge_dst(lib, rng, n=10)
    fails += pins.pin_negatives(lib, rng, n=30)
    fails += pins.pin_edge_blocks(lib, rng, n=25)
    fails += pins.pin_edge_errors(lib)
    fails += pins.pin_layer_draw(lib, rng, n=30)
    fails += pins.pin_layer_weight(lib, rng, n=30)
    fails += pins.pin_layer_blocks(lib, rng, n=25)
    fails += pins.pin_layer_errors(lib)
    fails += pins.pin_layer_boundaries(lib, n_draw=8)
    return fails


@pytest.mark.parametrize("label,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, label, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site for '{label}' not found once"
    src = tmp_path / "oracle_mutant.c"
    src.write_text(text.replace(old, new))
    so = str(tmp_path / "liboracle_mutant.so")
    oracle.build(so, extra_flags=("-w",), src=str(src))
    # in a child process: a mutant that corrupts memory crashes it, which also
    # counts as caught
    code = ("import sys; sys.path[:0] = [%r, %r]; import oracle, test_oracle_mutants as m; "
            "f = m.fast_pins(oracle.load(%r)); print('FAILS', len(f)); "
            "print(chr(10).join(f[:3]))" % (ROOT, HERE, so))
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         timeout=600)
    caught = res.returncode != 0 or "FAILS 0" not in res.stdout
    assert caught, f"no pin caught the mutant '{label}'"


def test_unmutated_passes_fast_pins():
    oracle.build()
    assert not fast_pins(oracle.load())
