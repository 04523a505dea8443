"""Former callables for the serving loop: the oracle (pure Python) and the
C++ library, both returning the same plan dict."""

import dataclasses

import numpy as np

from oracle import former as of


def oracle_former(params: of.Params, block_size: int = 16):
    def run(recs, free_blocks, now):
        reqs = [of.Request(**r) for r in recs]
        p = of.form_batch(reqs, free_blocks, block_size, now, params)
        return dict(budget=p.budget, ids=p.ids, q_len=p.q_len, theta=p.theta, resume_ids=p.resume_ids,
                    park_ids=p.park_ids, free_ids=p.free_ids, policy=p.policy, cost=p.cost)
    return run


def library_former(params: of.Params, block_size: int = 16):
    import paper_2512_04013_amd as aug
    cp = aug.former_params(beta=params.beta, t_max=params.t_max, beta_low=params.beta_low,
                           beta_high=params.beta_high, chunk_cap=params.chunk_cap, t_iter=params.t_iter,
                           fwd_a=params.fwd_a, fwd_b=params.fwd_b, swap_s_per_tok=params.swap_s_per_tok,
                           n_fwd_max=params.n_fwd_max, skip_instead_of_break=params.skip_instead_of_break,
                           block_size=block_size, order=params.order)

    def run(recs, free_blocks, now):
        arr = np.zeros(len(recs), aug.REQUEST_DTYPE)
        for i, r in enumerate(recs):
            for k, v in r.items():
                arr[i][k] = v
        return aug.aug_form_batch(arr, free_blocks, now, cp)
    return run


def lockstep(oracle, library):
    """A former that runs both and insists on identical plans (theta bit for bit)."""
    def run(recs, free_blocks, now):
        a = oracle(recs, free_blocks, now)
        b = library(recs, free_blocks, now)
        assert a["budget"] == b["budget"]
        assert list(a["ids"]) == list(b["ids"]), (now, a["ids"][:8], list(b["ids"][:8]))
        assert list(a["q_len"]) == list(b["q_len"])
        assert np.array_equal(np.array(a["theta"], np.float64).view(np.uint64),
                              np.asarray(b["theta"], np.float64).view(np.uint64))
        for k in ("resume_ids", "park_ids", "free_ids", "policy"):
            assert list(a[k]) == list(b[k]), k
        return b
    return run


class OracleLifecycle:
    """Request-record transitions of the oracle (Algorithm 1, steps (1)-(2))."""

    def arrive(self, **kw):
        return dataclasses.asdict(of.arrive(**kw))

    def on_return(self, rec, **kw):
        return dataclasses.asdict(of.on_return(of.Request(**rec), **kw))


class LockstepLifecycle:
    """Both lifecycles on every event; records must agree bit for bit."""

    def __init__(self):
        import paper_2512_04013_amd.runtime as rt
        self.a, self.b = OracleLifecycle(), rt.serving_lifecycle()

    @staticmethod
    def _same(x, y):
        assert set(x) == set(y)
        for k in x:
            if isinstance(x[k], float) or isinstance(y[k], float):
                assert np.float64(x[k]).view(np.uint64) == np.float64(y[k]).view(np.uint64), k
            else:
                assert x[k] == y[k], (k, x[k], y[k])

    def arrive(self, **kw):
        x, y = self.a.arrive(**kw), self.b.arrive(**kw)
        self._same(x, y)
        return y

    def on_return(self, rec, **kw):
        x, y = self.a.on_return(dict(rec), **kw), self.b.on_return(dict(rec), **kw)
        self._same(x, y)
        return y
