"""The MISA-T controller replay driving the library on the GPU: admissions, prompt and turn prefills,
decode steps with group-prefix hints, page reuse after completions and evictions, over one pool.  Every
kernel must exit cleanly (no device-side error), and the last decode step must match the oracle over the
K/V that kv_gather reads back from the pool for those sessions."""
import numpy as np
import pytest

import oracle
from misa_t.engine import LibraryEngine
from misa_t.replay import Replay, ReplayConfig
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

from gpu_helpers import assert_close, note, oracle_by_kv_head

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("policy", ["space", "time"])
def test_replay_on_the_library(policy):
    import torch
    cfg = ReplayConfig(steps=120, pool_pages=2048, length_scale=1.0 / 32, seed=11, max_outstanding=48)
    eng = LibraryEngine(cfg, keep_last=True, seed=3)
    r = Replay(cfg, policy=policy, engine=eng)
    note(f"misa_t replay {policy}: {cfg.steps} steps")
    m = r.run()
    torch.cuda.synchronize()
    assert eng.pool.device_error() == kp.KVP_OK
    assert min(eng.calls.values()) > 0 and sum(m["completed"].values()) > 20
    q, out, bt, lens = eng.last_decode
    pick = list(range(min(6, len(lens))))
    k, v = kp.kv_gather(eng.pool, 0, bt[pick].contiguous(), lens[pick])
    kb, vb = W.to_numpy_bits(k), W.to_numpy_bits(v)
    qb = W.to_numpy_bits(q)
    off, ref = 0, []
    for i in pick:
        n = int(lens[i])
        ref.append(oracle_by_kv_head(oracle.decode_seq, qb[i], kb[off:off + n], vb[off:off + n], 1.0 / np.sqrt(cfg.d)))
        off += n
    assert_close(out[pick].float().cpu().numpy().astype(np.float64), np.stack(ref), f"replay {policy} last decode")
    note(f"misa_t replay {policy}: {m['completed']} completed, hit rate {m['hit_rate']:.3f}, calls {eng.calls}")
    eng.close()
