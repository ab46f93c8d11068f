"""The closed serving loop on the GPU, checked end to end against the fp64
oracle: the C++ scheduler's batches drive the HIP step round after round
(slots taken and reused, chunks at increasing offsets, decode rows); the
K/V pools after the last round must equal, bit for bit, the oracle's
replay of every round's append, and the last round's attention output
must match the oracle's attention over those pools."""

import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from gpu_util import MAX_ABS, MEAN_ABS, say
from paper_2606_09061_amd import sched, serve

pytestmark = pytest.mark.gpu


class Recorder:
    def __init__(self, eng):
        self.eng = eng
        self.rounds = []

    def step(self, rows):
        self.rounds.append(np.array(rows, dtype=np.int32).reshape(-1, 4))
        return self.eng.step(rows)


def _words(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("chunking", [sched.CHUNK_TOKEN_BUDGET, sched.CHUNK_LPRS])
def test_closed_loop_pools_and_last_round_match_oracle(chunking):
    hq, hkv, d, bsz, slots, max_len = 4, 2, 64, 16, 6, 512
    say(f"closed loop chunking={chunking}")
    eng = serve.StepEngine(hq=hq, hkv=hkv, d=d, bsz=bsz, max_seqs=slots, max_seq_len=max_len,
                           max_tokens=256, seed=3)
    kc0, vc0 = _words(eng.kc).copy(), _words(eng.vc).copy()
    rec = Recorder(eng)
    reqs = wl.uniform_stream(24, 30.0, seed=5, max_seq_len=max_len, prompt_median=60,
                             output_median=6)
    cfg = sched.make_config(max_tokens=96, max_seqs=slots, max_seq_len=max_len, chunking=chunking,
                            target_us=30.0, delta=16, apc=chunking == sched.CHUNK_LPRS,
                            max_active=2, min_chunk=8)

    class Linear:  # a fixed linear latency model for LPRS (only its decisions matter here)
        def load_into(self, s):
            w = np.zeros((1, 16))
            w[0, 12] = 0.2
            s.set_predictor([(w, np.array([10.0]))], np.zeros(16), np.ones(16), 1.0)

    res = serve.serve(cfg, reqs, rec, predictor=Linear() if chunking == sched.CHUNK_LPRS else None,
                      memory_features=False)
    torch.cuda.synchronize()
    assert res["requests"] == 24 and len(rec.rounds) == res["rounds"] > 10
    # slots were reused: more requests than slots went through
    assert len(reqs) > slots
    bt = eng.bt.cpu().numpy()
    nb = bt.size
    kc, vc = kc0, vc0
    kn, vn = eng.kn.cpu(), eng.vn.cpu()
    batch = None
    for rows in rec.rounds:
        T = int(rows[:, 2].sum())
        batch = wl.Batch("round", hq, hkv, d, bsz, rows, bt, nb, 0)
        kc, vc = oracle.kv_append(batch, kn[:T], vn[:T], kc, vc)
    assert np.array_equal(_words(eng.kc).reshape(-1), kc.reshape(-1)), "K pool differs"
    assert np.array_equal(_words(eng.vc).reshape(-1), vc.reshape(-1)), "V pool differs"
    T = int(batch.rows[:, 2].sum())
    ref = oracle.attn(batch, eng.q[:T].cpu(), kc, vc)
    got = eng.out[:T].float().cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    say(f"last round: {batch.n_rows} rows, T={T}, max {err.max():.3e} mean {err.mean():.3e}")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS
