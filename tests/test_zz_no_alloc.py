"""The allocation-free prefix call against the workspace one (GPU).

tts_prefix_decode_attn_noalloc runs the same kernels and plan as
tts_prefix_decode_attn with its partial states in the library's own 64 MiB
scratch array, so its rows must equal the workspace call's bit for bit (and
meet the oracle's tolerance). Two calls in a row on one GPU, the second with
a smaller batch, exercise the shared array across calls; a plan that needs
more than the array holds is refused before anything is enqueued.
"""

import numpy as np
import pytest
import torch

from oracle.attention import oracle_attn_workload
from paper_2509_00195_amd import TTSError, tts_prefix_decode_attn_noalloc, tts_prefix_decode_workspace_size
from paper_2509_00195_amd.runner import PrefixAttention
from paper_2509_00195_amd.tts import TTS_ERR_WORKSPACE
from tts_synth import make_workload
from tts_synth.device import to_device

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20
TOL = {"f32": 1e-4, "bf16": 1e-2, "fp8": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    torch.cuda.set_device(0)


def _noalloc(pref, x, wl, out):
    tts_prefix_decode_attn_noalloc(pref.desc, pref.meta, x.q, x.k_cache, x.v_cache, x.k_scale, x.v_scale,
                                   x.block_tables, int(x.block_tables.shape[1]), x.seq_lens, wl.num_blocks, out)


def test_noalloc_equals_workspace_call_twice():
    for name, seed in [("7b64", 0), ("1p5b16", 1)]:  # the second call's batch is smaller
        wl = make_workload(name, seed)
        x = to_device(wl)
        pref = PrefixAttention(x, wl.req_seq_offsets, wl.block_tables, wl.seq_lens, wl.num_blocks)
        assert 0 < pref.ws_bytes <= SCRATCH_BYTES
        ref = pref().clone()
        out = torch.full_like(ref, float("nan"))
        _noalloc(pref, x, wl, out)
        torch.cuda.synchronize()
        print(f"noalloc {name}: workspace {pref.ws_bytes} bytes", flush=True)
        assert torch.equal(out, ref)
        err = float(np.max(np.abs(out.cpu().numpy().astype(np.float64) - oracle_attn_workload(wl))))
        assert err <= TOL[wl.shape.kv_dtype]


def test_noalloc_refuses_a_plan_beyond_its_scratch():
    """12,288 single-beam requests of one block at the 7B shape: 28 partial rows per beam of
    2 * 128 + 16 bytes, about 94 MB, more than the 64 MiB the call holds."""
    from paper_2509_00195_amd.runner import desc_for
    from tts_synth import AttnShape

    n = 12288
    sh = AttnShape(28, 4, 128, 16, "bf16", "bf16")
    offs = np.arange(n + 1, dtype=np.int32)
    tables = np.arange(n, dtype=np.int32).reshape(n, 1)
    lens = np.full(n, 16, np.int32)
    from paper_2509_00195_amd import tts_build_prefix_meta

    desc = desc_for(sh)
    meta = tts_build_prefix_meta(offs, tables, lens, 16, n, desc=desc)
    assert tts_prefix_decode_workspace_size(desc, meta) > SCRATCH_BYTES
    dev = torch.device("cuda:0")
    q = torch.zeros((n, 28, 128), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((n, 4, 16, 128), dtype=torch.bfloat16, device=dev)
    v = torch.zeros((n, 4, 128, 16), dtype=torch.bfloat16, device=dev)
    t = torch.from_numpy(tables).to(dev)
    ln = torch.from_numpy(lens).to(dev)
    out = torch.zeros((n, 28, 128), dtype=torch.float32, device=dev)
    with pytest.raises(TTSError) as e:
        tts_prefix_decode_attn_noalloc(desc, meta, q, k, v, None, None, t, 1, ln, n, out)
    assert e.value.status == TTS_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0  # nothing was enqueued
