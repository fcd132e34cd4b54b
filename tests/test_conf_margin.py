"""The confidence margin rule, on the CPU (App. B.2: the streak counts steps whose confidence exceeds
theta_conf = 0.9, a strict float32 comparison that decides an integer).

The oracle follows every sequence that a GPU parity test follows, and all 32 sequences x 128
steps of the benchmark workload. At every step its confidence c(t) must lie more than 0.018 from
0.9 (outside [0.882, 0.918]), far above the 2e-4 confidence tolerance of the parity tests (which
bounds the two paths' confidence difference), so both paths take the same streak decision and a
bit-exact comparison of decisions is meaningful. A workload whose seed fails is bumped by 1000
(tests/golden/conf_margins.py keeps the count; the benchmark workload needed nine bumps). The
record stored by that script must be reproduced exactly.
"""
import os

from golden import conf_margins as cm


def test_confidence_margins_of_every_followed_sequence():
    rows = cm.run(cm.jobs(), min(8, os.cpu_count() or 1))
    stored = {(r[0], r[1]): r for r in cm.read()}
    assert len(rows) == sum(len(w[3]) for w in cm.WORKLOADS) == len(stored)
    for name, b, steps, dmin, near, band in rows:
        assert band == 0 and near == 0 and dmin > cm.BAND, (name, b, dmin)
        s = stored[(name, b)]
        assert s[2] == steps and s[4] == near and s[5] == band, (name, b)
        assert abs(s[3] - dmin) <= 1e-12 * max(1.0, dmin), (name, b, s[3], dmin)
    bench = [r for r in rows if r[0].startswith("7b-b32")]
    assert sorted(r[1] for r in bench) == list(range(32)) and all(r[2] == 128 for r in bench)
    assert cm.SEED_BUMPS.get("7b-b32 (benchmark)") == 9
