"""Workloads for the tests: the seeded generator's arrays plus completion
events whose admission estimates come from the CPU oracle's score stage
(state 1: the B-free estimate), so that no input of either side is computed
by the generator or by the HIP path."""
import numpy as np

import oracle
import workloads


def est_base(b):
    """The B-free admission estimate of every request (oracle score with all
    factors 1, counts = the generator's word counts)."""
    return oracle.score(b.words, b.category, b.tenant, b.group, b.t_base, b.s_tenant,
                        np.ones(b.n_groups), f_ref=b.f_ref)[0]


def load(name, n=None, with_text=True):
    b = workloads.generate(name, n=n, with_text=with_text)
    return workloads.complete(b, est_base(b))
