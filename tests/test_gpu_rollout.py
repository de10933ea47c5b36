"""The rollout pipeline (Acquire -> Run -> Eval worker pools around the
continuous-batching engine) on the GPU: every trajectory it produces, under
a coupled and a decoupled setting, is checked token by token against the
reference trajectory (its whole history as one causal prefill through the
reference layers, then the reference head with the same draws), and every
page returns to the pools."""
import numpy as np
import pytest
import torch

from oracle import generate as OG
from oracle import oracle as O
from paper_2608_22167_amd import rollout as R, workload as W
from paper_2608_22167_amd.generate import GenSpec, Generator
from tests.test_gpu_generate import DELTA

pytestmark = pytest.mark.gpu


def test_pipeline_trajectories_match_reference():
    torch.cuda.set_device(0)
    base = W.replace(W.GPT_OSS_20B, hidden=256, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                     ffn_dim=256)
    spec = GenSpec(n_layers=4, base=base, vocab=4096, window=128, pages_full=1024, pages_sw=256, max_ctx=4096,
                   seed=3101)
    gen = Generator(spec, max_tokens_per_step=1024)
    free0 = gen.free_pages()
    common = dict(n_trajectories=12, eval_workers=2, turns=3, tokens_per_turn=5, prompt_tokens=(10, 120),
                  obs_tokens=(5, 40), acquire_s=(0.01, 0.03), tool_s=(0.02, 0.06), eval_s=(0.0, 0.01),
                  vocab=spec.vocab)
    runs = {}
    for name, aw, rw in (("coupled", 3, 3), ("decoupled", 3, 8)):
        eng = R.Engine(gen)
        try:
            res = R.run_pipeline(R.RolloutConfig(acquire_workers=aw, run_workers=rw, in_flight=8, **common), eng)
        finally:
            eng.close()
        assert gen.free_pages() == free0, "pages leaked"
        assert gen.check_errors() == 0
        runs[name] = res
        print(f"  {name}: {res['tokens']} tokens in {res['wall_s']:.2f} s, mean batch {res['mean_batch']:.1f}, "
              f"engine busy {res['engine_busy']:.2f}")
    ss = spec.stack_spec()
    lw = [W.stack_weights_host(ss, i) for i in range(spec.n_layers)]
    lm = W.lm_weights_host(spec.seed, ss.shape_full.hidden, spec.vocab)
    same = 0
    for tid in range(common["n_trajectories"]):
        for name, res in runs.items():
            rec = res["records"][tid]
            assert len(rec.sampled) == common["turns"] * common["tokens_per_turn"]
            rows = OG.trajectory_rows(ss, lw, lm["embed"], rec.tokens[:-1])
            pos = np.array([p for p, _, _ in rec.sampled])
            ref = O.lm_head(rows[pos - 1], lm["g_final"], lm["w_lm"], ss.shape_full.rms_eps, spec.temperature,
                            seed=spec.seed, seq_ids=np.full(len(pos), tid, np.int32), positions=pos,
                            want_logits=True)
            for i, (p, tok, lp) in enumerate(rec.sampled):
                best = int(ref["tokens"][i])
                if tok != best:
                    sc = ref["pert"][i]
                    assert sc[best] - sc[tok] <= DELTA, (name, tid, p, tok, best)
                else:
                    assert abs(lp - ref["logprob"][i]) <= 2e-3
        same += runs["coupled"]["records"][tid].tokens == runs["decoupled"]["records"][tid].tokens
    print(f"  {same} of {common['n_trajectories']} trajectories identical under both settings")
