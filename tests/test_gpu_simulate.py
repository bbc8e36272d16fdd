"""The acceptance simulation harness (paper_2601_09083_amd/simulate.py) on a
small GRPO-shaped group: every strategy and drafting variant runs the loop
through libsrt, and every committed token must be the sequence's true
continuation (checked inside run()); accepted counts are bounded by the
drafted nodes."""
import pytest

from paper_2601_09083_amd import simulate as SIM
from paper_2601_09083_amd import workload as W
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

CFG = W.Config("sim_small", 8, n_prompts=4, seqs_per_prompt=4, vocab=4096, rollouts_per_prompt=8,
               rollout_len=W.Dist("uniform", 400, 1200), ctx_len=W.Dist("uniform", 200, 800), n_nodes=32,
               max_depth=8, hq=4, hkv=1, head_dim=64)


@pytest.mark.parametrize("strategy,variant", [("history", {}), ("onthefly", {}), ("runahead", {}),
                                              ("onthefly", {"chain": True, "n_nodes": 9}),
                                              ("onthefly", {"min_score": 0.1}), ("onthefly", {"alpha": 2.0})])
def test_simulation_loop(strategy, variant):
    steps = 12
    say(f"simulate: {strategy} {variant}")
    sim = SIM.make_sim_tokens(CFG, future_len=(steps + 2) * (CFG.max_depth + 1), runahead_per_prompt=2)
    r = SIM.run(CFG, sim, steps, strategy, **variant)
    assert 0.0 <= r["mean_accepted_per_step"] <= r["mean_tree_nodes"] - 1.0 + 1e-9
    assert r["mean_emitted_per_step"] == pytest.approx(r["mean_accepted_per_step"] + 1.0)
    assert r["mean_accepted_per_step"] > 0.2, "drafts from mutated rollouts should often be accepted"
