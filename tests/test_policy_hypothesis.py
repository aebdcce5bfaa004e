"""Property-based parity of the library's scaling policy with the oracle:
hypothesis draws parameters, batches and horizons; every output must match
bit for bit (host code, no GPU)."""
import math

from hypothesis import HealthCheck, given, settings, strategies as st

from oracle import kf_policy as O
from paper_2606_29207_amd import policy as L

from test_policy_parity import FIELDS, compare_sim

params = st.fixed_dictionaries(dict(
    num_kv_heads=st.integers(1, 4), head_dim=st.integers(1, 8), num_layers=st.integers(1, 4),
    elem_bytes=st.sampled_from([1, 2]),
    beta_mem=st.floats(0.05, 1.0), beta_slo=st.floats(0.05, 1.0), gamma=st.floats(0.05, 1.0),
    t_a_max=st.floats(0.01, 10.0), bw_hbm=st.floats(1.0, 1e3), c_kv_cap=st.floats(10.0, 1e4),
    t_step=st.floats(0.01, 5.0), t_prewarm=st.floats(0.0, 20.0)))


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(p=params, lens=st.lists(st.integers(0, 200), max_size=8),
       gens=st.lists(st.integers(0, 60), max_size=8), steps=st.integers(0, 70))
def test_policy_library_matches_oracle(p, lens, gens, steps):
    gens = (gens + [0] * len(lens))[:len(lens)]
    need = math.ceil(sum(lens) * O.token_bytes(p) / O.threshold(p)[0])
    if need > 20000:        # keep the brute-force oracle quick
        return
    pl = L.params(**{k: p[k] for k in FIELDS})
    assert L.threshold(pl) == O.threshold(p)
    compare_sim(p, pl, lens, gens, steps)
