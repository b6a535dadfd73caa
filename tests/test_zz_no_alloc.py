"""mx_paged_attn_static: the attention entry point that allocates nothing (its
metadata and split partials live in the library's static device scratch)
against mx_paged_attn, the entry point it varies, on two calls in a row, the
second with a smaller batch, so that the second call runs over what the first
left in the shared scratch; both also against the oracle.  Plus the host-side
rejection of a batch that needs more scratch than the array holds."""
import sys

import numpy as np
import pytest

import workload as wl
from helpers import assert_rows_close, bits_to_f64, mx_batch, mx_shape

torch = pytest.importorskip("torch")
import paper_2606_16264_amd as mx  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_static_rejects_batches_beyond_the_scratch():
    """Host-side check, before any device work (this also runs without a
    GPU): a batch whose page tables alone exceed the static scratch."""
    cap = mx.mx_paged_attn_static_max_bytes()
    assert cap == 32 << 20
    n_pages = cap // 4 + 16
    ctx = 16 * n_pages - 16
    pages = np.arange(n_pages, dtype=np.int32)
    b = mx.Batch([mx.MX_DECODE], [1], [ctx], [pages])
    shape = mx.attn_shape(8, 1, 128, n_pages)
    st = mx.lib().mx_paged_attn_static(b.ptr, mx.ctypes.byref(shape), 0x1000, 0x2000, 0x3000,
                                       0x4000, None)
    assert st == mx.MX_ERR_TOO_LARGE
    assert "static scratch" in mx.last_error()
    st = mx.lib().mx_paged_attn_static(b.ptr, mx.ctypes.byref(shape), None, 0x2000, 0x3000,
                                       0x4000, None)
    assert st == mx.MX_ERR_NULL


def _case(cfg, b, seed, rng):
    # imported here: the GPU parity module skips itself without a GPU
    from test_gpu_parity import attention_case
    return attention_case(cfg, b, seed, rng)


@pytest.mark.gpu
def test_static_matches_workspace_entry_point_twice():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = wl.LayerConfig("t", 256, 256, 32, 8, 128)
    rng = np.random.default_rng(71)
    # first call: few long decodes (several key splits each, so partials and
    # merges), prefill chunks with and without a cached prefix; second call:
    # a smaller batch with fewer, shorter requests
    big = wl.custom_batch(rng, [9000, 16383, 4097, 30, 700], [(300, 0), (129, 511)])
    small = wl.custom_batch(rng, [5000, 17], [(40, 16)])
    cases = [("big", big), ("small", small)]
    for name, b in cases:
        say(f"case: static attention, {name} batch T={b.T} R={b.R}")
        c = _case(cfg, b, 21, rng)
        ref = torch.empty((b.T, cfg.n_q_heads, cfg.head_dim), dtype=torch.uint16, device="cuda")
        mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], ref, c["ws"])
        got = torch.full_like(ref, 0x7FC1)
        mx.mx_paged_attn_static(c["mb"], c["shape"], c["q"], c["k"], c["v"], got)
        torch.cuda.synchronize()
        # same kernels and the same plan: bit for bit
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), name
        n = b.T * cfg.n_q_heads
        assert_rows_close(bits_to_f64(got).reshape(n, -1), c["exp"].reshape(n, -1),
                          what=f"static attention ({name})")
        say(f"  {name}: bit-identical to mx_paged_attn, within 2e-2 of the oracle")
