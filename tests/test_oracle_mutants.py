"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pins catch every one of them.

Each mutant is a one-token edit of ``oracle/oracle.cpp`` (a dropped term, a
wrong sign or index, a swapped operand, a flipped comparison); it is built
into a temporary library and the pin suite is run against it in a child
process.  A mutant the pins do not kill would mean the oracle could carry
that mistake unnoticed.
"""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.cpp")

MUTANTS = [
    ("drop the N*C term", "a[2] * N * C", "0.0 * N * C"),
    ("C term uses N", "a[4] * C", "a[4] * N"),
    ("N^2 term uses C", "a[3] * N * N", "a[3] * C * C"),
    ("W sign", "t_prefill(m, (double)c.n, (double)c.c) - tpf_cached", "t_prefill(m, (double)c.n, (double)c.c) + tpf_cached"),
    ("no clamp of W", "std::max(0.0, t_prefill(m, (double)c.n, (double)c.c) - tpf_cached)", "(t_prefill(m, (double)c.n, (double)c.c) - tpf_cached)"),
    ("Z without cached term", "const double Z = tpf_cold - tpf_cached;", "const double Z = tpf_cold;"),
    ("rho strict", "c.inC = c.rho <= m.eta;", "c.inC = c.rho < m.eta;"),
    ("Z<=0 ignored", "if (!kvc_on || Z <= 0.0) {", "if (!kvc_on) {"),
    ("tpot non-strict", "c.tpot < m.tau", "c.tpot <= m.tau"),
    ("interference always", "active > 0 ? tpf", "active >= 0 ? tpf"),
    ("interference not amortised", "tpf / std::max(1.0, m.lout)", "tpf"),
    ("segment exclusive", "if (B <= m.seg_ub[s]) return s;", "if (B < m.seg_ub[s]) return s;"),
    ("gamma dropped", "m.gamma[s] * (m.beta[s][0]", "1.0 * (m.beta[s][0]"),
    ("B+ without arrival", "const int64_t Bp = active + 1;", "const int64_t Bp = active;"),
    ("S+ without request", "const double Sp = (double)(sn.S[i] + L);", "const double Sp = (double)(sn.S[i]);"),
    ("TTFT queue uses Q for P", "m.alpha[1] * (double)sn.P[i]", "m.alpha[1] * (double)sn.Q[i]"),
    ("SLO from cached prefill", "std::max(m.ttft_floor, tpf_cold)", "std::max(m.ttft_floor, tpf_cached)"),
    ("D order", "default:  // SEL_DCQ\n        if (Da != Db) return Da > Db;", "default:  // SEL_DCQ\n        if (Da != Db) return Da < Db;"),
    ("hit order", "default:  // SEL_DCQ\n        if (Da != Db) return Da > Db;\n        if (a.hit != b.hit) return a.hit > b.hit;", "default:  // SEL_DCQ\n        if (Da != Db) return Da > Db;\n        if (a.hit != b.hit) return a.hit < b.hit;"),
    ("Q order", "if (a.hit != b.hit) return a.hit > b.hit;\n        if (Qa != Qb) return Qa < Qb;\n        break;\n    }", "if (a.hit != b.hit) return a.hit > b.hit;\n        if (Qa != Qb) return Qa > Qb;\n        break;\n    }"),
    ("id order", "return a.i < b.i;\n  };", "return a.i > b.i;\n  };"),
    ("LMetric without arrival", "* (unsigned __int128)(uint64_t)(active + 1);", "* (unsigned __int128)(uint64_t)(active);"),
    ("LMetric ignores n", "(uint64_t)(sn.P[c.i] + c.n)", "(uint64_t)(sn.P[c.i])"),
    ("capacity batch bound", "if (active + 1 <= m.b_max && sn.S[i] + L <= m.kv_cap)", "if (active + 1 < m.b_max && sn.S[i] + L <= m.kv_cap)"),
    ("capacity ignores tokens", "if (active + 1 <= m.b_max && sn.S[i] + L <= m.kv_cap)", "if (active + 1 <= m.b_max && sn.S[i] <= m.kv_cap)"),
    ("walk skips last block", "while (j < ch.len() && set.count(ch.at(j)) != 0) ++j;", "while (j + 1 < ch.len() && set.count(ch.at(j)) != 0) ++j;"),
    ("walk past misses", "while (j < ch.len() && set.count(ch.at(j)) != 0) ++j;", "for (int32_t k = 0; k < ch.len(); ++k) j += set.count(ch.at(k)) != 0;"),
    ("cached tokens per block", "c.c = c.hit * m.block_tokens;", "c.c = c.hit;"),
    ("ttft miss non-strict", "if (best->ttft > slo) d.flags |= R_TTFT_MISS;", "if (best->ttft >= slo) d.flags |= R_TTFT_MISS;"),
    ("commit P counts cached", "sn.P[i] += L - hitb * block_tokens;", "sn.P[i] += L;"),
    ("D-Q queued order", "if (Qa != Qb) return Qa < Qb;\n        break;\n      case SEL_DC:", "if (Qa != Qb) return Qa > Qb;\n        break;\n      case SEL_DC:"),
    ("H-C-Q headroom direction", "if (ha != hb) return ha < hb;", "if (ha != hb) return ha > hb;"),
    ("random k from low bits", "const uint64_t k = ((z >> 32) * (uint64_t)d.nT) >> 32;", "const uint64_t k = z % (uint64_t)d.nT;"),
    ("D-C-Q fallback over A", "if (c.inC && (!best || before(SEL_DCQ, c, *best))) best = &c;", "if ((!best || before(SEL_DCQ, c, *best))) best = &c;"),
    ("LMetric selector order", "if (la != lb) return la < lb;", "if (la != lb) return la > lb;"),
    ("EMA weight", "const double w = 0.02;", "const double w = 0.2;"),
    ("EMA ratio clip", "ratio = std::min(2.0, std::max(0.5, ratio));", "ratio = std::min(4.0, std::max(0.5, ratio));"),
    ("EMA factor floor", "m->gamma[s] = std::min(2.0, std::max(1.0, f));", "m->gamma[s] = std::min(2.0, std::max(0.5, f));"),
    ("upper median", "m->lout = (double)recent[(cnt - 1) / 2];", "m->lout = (double)recent[cnt / 2];"),
    ("first token keeps pending", "P[i] -= tokens[k];", "P[i] -= 0;"),
    ("commit ignores cap", "if ((int64_t)set.size() < sn.cap) set.insert(key);", "if (true) set.insert(key);"),
    ("schedule without commit", "if (place >= 0) (void)commit_one(sn, ch, place, m->block_tokens, drop);", "(void)0;"),
    ("commit keeps the queue", "sn.Q[i] += 1;", "sn.Q[i] += 0;"),
    ("replay measures after commit",
     "    candidate_latency(sn, *m, i, L - c, c, L, tpot[k], ttft[k]);\n    hit[k] = (int32_t)hb;\n    (void)commit_one(sn, ch, i, m->block_tokens, drop);",
     "    (void)commit_one(sn, ch, i, m->block_tokens, drop);\n    candidate_latency(sn, *m, i, L - c, c, L, tpot[k], ttft[k]);\n    hit[k] = (int32_t)hb;"),
    ("replay hit after commit", "const int64_t hb = prefix_hit(sn.sets[(size_t)i], ch);", "const int64_t hb = ch.len();"),
    # the near-boundary rule (what the GPU parity check may skip)
    ("NB_TPOT window widened", "std::fabs(c.tpot - m.tau) <= NB_REL * m.tau;", "std::fabs(c.tpot - m.tau) <= 10 * NB_REL * m.tau;"),
    ("NB_TPOT never raised", "std::fabs(c.tpot - m.tau) <= NB_REL * m.tau;", "std::fabs(c.tpot - m.tau) < 0.0;"),
    ("NB_TPOT always raised", "const bool tpot_near = !(m.flags & F_NO_TPOT) &&", "const bool tpot_near = true ||"),
    ("NB_TPOT over all of A", "c.unsure = c.inC && (", "c.unsure = ("),
    ("every unsure candidate decides", "const bool decides = sel == SEL_RANDOM", "const bool decides = true || sel == SEL_RANDOM"),
    ("only the choice decides", "&c == best ||\n                         (!c.inT && (!best || before(sel, c, *best)));", "&c == best;"),
    ("unsure count not reported", "d.nb |= std::min<uint32_t>(n_unsure, 0xFFFFu) << 16;", "(void)n_unsure;"),
    ("NB_TTFT window widened", "std::fabs(c.ttft - slo) <= NB_REL * slo;", "std::fabs(c.ttft - slo) <= 10 * NB_REL * slo;"),
    ("NB_TTFT never raised", "std::fabs(c.ttft - slo) <= NB_REL * slo;", "std::fabs(c.ttft - slo) < 0.0;"),
    ("NB_TTFT on TTFT equal to the budget", "(m.flags & F_TTFT_ADMIT) && !ttft_is_budget(c) &&", "(m.flags & F_TTFT_ADMIT) &&"),
    ("NB_MISSFLAG window widened", "std::fabs(best->ttft - slo) <= NB_REL * slo) d.nb |= NB_MISSFLAG;", "std::fabs(best->ttft - slo) <= 10 * NB_REL * slo) d.nb |= NB_MISSFLAG;"),
    ("NB_MISSFLAG never raised", "std::fabs(best->ttft - slo) <= NB_REL * slo) d.nb |= NB_MISSFLAG;", "std::fabs(best->ttft - slo) < 0.0) d.nb |= NB_MISSFLAG;"),
    ("NB_MISSFLAG on TTFT equal to the budget", "if (!ttft_is_budget(*best) && std::fabs", "if (std::fabs"),
    ("NB_RHO window widened", "std::fabs(c.rho - m.eta) <= NB_REL * std::max(m.eta, 1.0)", "std::fabs(c.rho - m.eta) <= 10 * NB_REL * std::max(m.eta, 1.0)"),
    ("NB_RHO on rho = 1 by construction", "const bool exact_one = some_full && c.c == 0;", "const bool exact_one = false;"),
    ("rho = 1 exemption without a full hit", "const bool exact_one = some_full && c.c == 0;", "const bool exact_one = c.c == 0;"),
    ("NB_RHO never raised", "std::fabs(c.rho - m.eta) <= NB_REL * std::max(m.eta, 1.0)", "std::fabs(c.rho - m.eta) < 0.0"),
    ("NB_Z window widened", "std::fabs(Z) <= NB_REL * std::fabs(tpf_cold)", "std::fabs(Z) <= 10 * NB_REL * std::fabs(tpf_cold)"),
    ("NB_Z never raised", "std::fabs(Z) <= NB_REL * std::fabs(tpf_cold)", "std::fabs(Z) < 0.0"),
    # following another implementation's near-boundary placements
    ("follow ignored", "      place = follow[r];", "      place = d.inst;"),
    ("follow at every request", "if (follow && (d.nb & NB_CHOICE) && follow[r] != d.inst)", "if (follow && follow[r] != d.inst)"),
    ("follow unchecked", "if (!eligible) return -1;", "(void)eligible;"),
]


def _run_mutant(tmp, k, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation target not found: {old!r}"
    mut = src.replace(old, new, 1)
    d = os.path.join(tmp, f"m{k}")
    os.makedirs(d)
    cpp = os.path.join(d, "oracle.cpp")
    so = os.path.join(d, "liboracle.so")
    with open(cpp, "w") as f:
        f.write(mut)
    subprocess.run(["g++", "-O1", "-std=c++17", "-fopenmp", "-shared", "-fPIC", "-o", so, cpp],
                   check=True, capture_output=True)
    env = dict(os.environ, PS_ORACLE_MUTANT_LIB=so, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode


def test_every_planted_mistake_is_caught():
    with tempfile.TemporaryDirectory() as tmp:
        with ThreadPoolExecutor(max_workers=6) as ex:
            codes = list(ex.map(lambda a: _run_mutant(tmp, *a),
                                [(k, old, new) for k, (_, old, new) in enumerate(MUTANTS)]))
    survivors = [MUTANTS[k][0] for k, rc in enumerate(codes) if rc == 0]
    assert not survivors, f"pins missed planted mistakes: {survivors}"
