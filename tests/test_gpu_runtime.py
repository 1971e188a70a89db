"""The KV probe on the GPU (Sec. 2.2, paragraph "KV probe"): it times the three
paths once per 64-token prefix bucket, decides by the oracle's rule on its own
timings, and answers later calls in the bucket from the stored verdict."""
import dataclasses

import pytest
import torch

import oracle
import paper_2606_09937_amd as rk
import workloads
from gpu_util import log

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_kv_probe_times_paths_and_stores_verdict_per_bucket(dtype):
    shape = dataclasses.replace(workloads.get("tiny").model, dtype=dtype)
    mw = workloads.make_model(shape, seed=51, device=DEV)
    B, s = 4, 8
    prefix = workloads.make_tokens(200, shape.vocab, seed=51, name="prefix", device=DEV)
    sfx = workloads.make_tokens(B * s, shape.vocab, seed=51, name="suffix", device=DEV).reshape(B, s).contiguous()
    probe = rk.KVProbe(3)
    log(f"[probe {dtype}] n=100 (bucket 1)")
    share, t, probed = probe.decide(mw, prefix[:100].contiguous(), sfx)
    torch.cuda.synchronize()
    log(f"[probe {dtype}] times full/prefix/suffix {t} share={share}")
    assert probed and all(x > 0 for x in t)
    assert share == oracle.kv_probe_share(*t)
    # another prefix length in the same bucket: the stored verdict, nothing timed
    share2, t2, probed2 = probe.decide(mw, prefix[:70].contiguous(), sfx)
    assert not probed2 and share2 == share and t2 == t
    assert probe.lookup(127) == (share, t) and probe.lookup(128) is None
    # a new bucket is timed again
    log(f"[probe {dtype}] n=130 (bucket 2)")
    share3, t3, probed3 = probe.decide(mw, prefix[:130].contiguous(), sfx)
    torch.cuda.synchronize()
    assert probed3 and share3 == oracle.kv_probe_share(*t3)
    assert probe.lookup(191) == (share3, t3)
