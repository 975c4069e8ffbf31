"""HIP graph capture of the attention calls: every replay matches the eager
call bit for bit.

The prefix-shared call (attention kernel + merge) and the paged baseline are
captured together on a side stream and replayed several times, with eager
work and synchronisations between the replays; each replay is compared with
the eager result (both paths are deterministic: a fixed merge order and no
float atomics). The configurations cover both merge kernels (up to and over
4096 rows) and both paged modes (direct output and split partials).
"""

import pytest
import torch

from paper_2509_00195_amd.runner import PagedAttention, PrefixAttention
from tts_synth import make_workload
from tts_synth.device import to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    torch.cuda.set_device(0)


@pytest.mark.parametrize("name", ["tiny", "1p5b16", "7b64", "7b_straggler"])
def test_graph_replay_matches_eager(name):
    wl = make_workload(name, 0)
    x = to_device(wl)
    s = torch.cuda.Stream()
    pref = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.num_blocks, stream=s)
    paged = PagedAttention(x, wl.max_seq_len, wl.num_blocks)
    out_x, out_p = torch.empty_like(pref.out), torch.empty_like(pref.out)
    pref(out=out_x, stream=s)
    paged(out=out_p, stream=s)
    torch.cuda.synchronize()
    want_x, want_p = out_x.clone(), out_p.clone()
    assert torch.isfinite(want_x).all() and torch.isfinite(want_p).all()

    gx, gp = torch.empty_like(out_x), torch.empty_like(out_p)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pref(out=gx, stream=s)
        paged(out=gp, stream=s)
    torch.cuda.synchronize()
    for rep in range(4):
        gx.fill_(float("nan"))
        gp.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print(f"{name} replay {rep}", flush=True)
        assert torch.equal(gx, want_x) and torch.equal(gp, want_p), rep
        pref(out=out_x, stream=s)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out_x, want_x)
