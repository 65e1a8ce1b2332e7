"""Pins of the router-recall measurement (CPU): the R = 1 router is the
oracle router itself (recall and capture exactly 1), and no router captures
more of P_oracle's mass than P_oracle's own top-k (capture <= 1)."""
import numpy as np

from router_recall import recall_table
from workload import Problem, Selection, Workload


def test_recall_of_the_oracle_router_is_one_and_capture_is_bounded():
    w = Workload("recall-small", Problem(1, 2, 2, 64, 8, 16, 16), Selection(0, 6), 6001)
    t = recall_table(w, 12, 6, pools=[(2, 2, 2), (1, 2, 2), (4, 4, 4)])
    rm, rmin, cm, cmin = t["routers"]["1x1x1"]
    assert rm == 1.0 and rmin == 1.0 and cm == 1.0 and cmin == 1.0
    for name, (rm, rmin, cm, cmin) in t["routers"].items():
        assert 0.0 <= rmin <= rm <= 1.0
        assert cm <= 1.0 + 1e-12 and cmin <= cm
        print(name, rm, cm)
