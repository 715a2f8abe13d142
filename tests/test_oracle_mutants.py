"""Mutation test of the reference model's pins (CPU only).

Each case plants one plausible mistake into a private copy of
``oracle/hbf_oracle.c`` (a dropped term, a wrong index, a transposed
operand, a reversed tie-break ...), builds it, and runs the pin suite
against it.  The pins must fail for every mutant; the unmodified source must
pass (that is ``test_oracle_pins.py`` itself).
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "hbf_oracle.c")

MUTANTS = {
    "die-ignores-busy-die": (
        "int64_t start = db[L.key] ? orc_max(issue[i], df[L.key]) : issue[i];\n    if (m->fifo",
        "int64_t start = issue[i];\n    if (m->fifo"),
    "channel-tie-reversed": (
        "if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;",
        "if (x->idx != y->idx) return x->idx < y->idx ? 1 : -1;"),
    "channel-uses-issue": (
        "int64_t start = cb[c] ? orc_max(dd[i], cf[c]) : dd[i];",
        "int64_t start = cb[c] ? orc_max(issue[i], cf[c]) : issue[i];"),
    "map-transposed": (
        "L.ch = (uint32_t)(dp % p->channels);\n  L.die = (uint32_t)((dp / p->channels) % p->dies_per_channel);",
        "L.die = (uint32_t)(dp % p->dies_per_channel);\n  L.ch = (uint32_t)((dp / p->dies_per_channel) % p->channels);"),
    "xfer-floor": (
        "unsigned __int128 q = (num + p->channel_bytes_per_s - 1) / p->channel_bytes_per_s;",
        "unsigned __int128 q = num / p->channel_bytes_per_s;"),
    "native-path-delayed": (
        "if (!in[i]) complete[i] = issue[i];",
        "if (!in[i]) complete[i] = issue[i] + tR;"),
    "range-end-inclusive": (
        "addr - m->ranges[r].base < m->ranges[r].bytes) return r;",
        "addr - m->ranges[r].base <= m->ranges[r].bytes) return r;"),
    "dev-page-base-dropped": (
        "return orc_locate(m, m->ranges[r].dev_page_base + (addr - m->ranges[r].base) / m->p.page_bytes);",
        "return orc_locate(m, (addr - m->ranges[r].base) / m->p.page_bytes);"),
    "plane-flag-ignored": (
        "if (p->flags & ORC_FLAG_PLANE_PARALLEL) L.key = L.key * p->planes_per_die + L.plane;",
        "if (p->flags & ORC_FLAG_PLANE_PARALLEL) L.key = L.key * p->planes_per_die;"),
    "unsorted-not-detected": (
        "if (i > 0 && issue[i] < issue[i - 1]) bad_order = 1;",
        "if (i > 1 && issue[i] < issue[i - 2]) bad_order = 1;"),
    "state-not-committed": (
        "memcpy(m->chan_free, cf, sizeof(int64_t) * p->channels);",
        "(void)cf;"),
    "refresh-quantum-free": (
        "      in[i] = 2;  /* in range, claims a quantum */\n      start += tQ;",
        "      in[i] = 2;  /* in range, claims a quantum */"),
    "refresh-done-at-read-end": (
        "m->qdone[f->id[f->head++]] = dd[i] - tR;",
        "m->qdone[f->id[f->head++]] = dd[i];"),
    "refresh-quantum-without-read": (
        "const int64_t tQ = tR + m->t_prog_ns;\n\n  int overflow",
        "const int64_t tQ = m->t_prog_ns;\n\n  int overflow"),
    "refresh-drain-ignores-clock": (
        "int64_t start = m->die_busy[k] ? orc_max(m->die_free[k], t_from) : t_from;",
        "int64_t start = t_from;"),
    "cache-prefetch-ignores-residency": (
        "      if (c->slot[p + k] >= 0) continue;\n",
        ""),
    "cache-prefetch-depth-short": (
        "for (int64_t k = 1; k <= c->degree && p + k < c->range_pages; k++) {",
        "for (int64_t k = 1; k < c->degree && p + k < c->range_pages; k++) {"),
    "cache-eviction-keeps-page": (
        "    c->slot[old] = -1;\n",
        ""),
    "cache-hit-not-counted-used": (
        "if (c->frame_pf[c->slot[p]]) { c->frame_pf[c->slot[p]] = 0; c->pf_used++; }",
        "if (c->frame_pf[c->slot[p]]) { c->frame_pf[c->slot[p]] = 0; }"),
    "blocking-register-freed-at-read-end": (
        "int64_t s0 = orc_max(issue[i], complete[best]);",
        "int64_t s0 = orc_max(issue[i], dd[best]);"),
    "blocking-channel-tie-reversed": (
        "(dd[i] == dd[best] && i < best)",
        "(dd[i] == dd[best] && i > best)"),
    "vmem-charges-whole-burst": (
        "int64_t service = orc_vmem_burst_ns(m, L) - orc_vmem_burst_ns(m, L - 1);",
        "int64_t service = orc_vmem_burst_ns(m, L);"),
    "vmem-reverse-continues": (
        "L = (have && page == last + 1) ? L + 1 : 1;",
        "L = (have && (page == last + 1 || page + 1 == last)) ? L + 1 : 1;"),
    "vmem-native-breaks-burst": (
        "if (r < 0) { complete[i] = issue[i]; continue; }\n    uint64_t page",
        "if (r < 0) { complete[i] = issue[i]; have = 0; continue; }\n    uint64_t page"),
    "vmem-tail-slope-from-wrong-segment": (
        "return T[5] + (int64_t)((__int128)(T[5] - T[4]) * (L - 512) / 256);",
        "return T[5] + (int64_t)((__int128)(T[5] - T[3]) * (L - 512) / 448);"),
    "vmem-route-never-busy": (
        "int64_t start = vb ? orc_max(issue[i], vf) : issue[i];",
        "int64_t start = issue[i];"),
    "vmem-interpolation-rounds-up": (
        "return T[s] + (int64_t)((__int128)(T[s + 1] - T[s]) * (L - La) / (Lb - La));",
        "return T[s] + (int64_t)(((__int128)(T[s + 1] - T[s]) * (L - La) + (Lb - La) - 1) / (Lb - La));"),
    "vmem-burst-state-not-kept": (
        "m->vfree = vf; m->vbusy = vb; m->vhave = have; m->vlast = last; m->vburst = L;",
        "m->vfree = vf; m->vbusy = vb; m->vhave = 0; m->vlast = last; m->vburst = L;"),
    "extra-service-term": (
        "complete[i] = start + xfer;",
        "complete[i] = start + xfer + (start > dd[i] ? 1 : 0);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/present: {name}"
    mut = tmp_path / "mutant.c"
    mut.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-std=gnu11", "-shared", "-fPIC", str(mut), "-o", str(lib), "-lm"])
    env = dict(os.environ, HBF_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_events.py"),
                        os.path.join(ROOT, "tests", "test_oracle_refresh.py"),
                        os.path.join(ROOT, "tests", "test_oracle_cache.py"),
                        os.path.join(ROOT, "tests", "test_oracle_blocking.py"),
                        os.path.join(ROOT, "tests", "test_oracle_vmem.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
