"""skipconv_step_static (no allocation; its scratch is a fixed device array in the
library) against skipconv_step of a layer handle with the same descriptor, split
pipeline and caller-retained frames: z bit-identical after every call. The calls
run in a row on one device, a larger layer first and a smaller one after it, so
the second call finds the first one's leftovers in the shared scratch."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2104_11487_amd import skipconv as S  # noqa: E402
from paper_2104_11487_amd import synthetic as syn  # noqa: E402
from parity_util import say, to_device, weight_storage  # noqa: E402

pytestmark = pytest.mark.gpu

# n, h, w, c_in, c_out, k, stride, groups, block, dtype, eps
CASES = [
    (2, 64, 48, 64, 64, 3, 1, 1, 8, "bf16", 1.2),    # block-halo MFMA convolution
    (1, 24, 20, 32, 32, 3, 1, 1, 4, "bf16", 0.9),    # smaller: block-halo, 4 x 4 blocks
    (1, 19, 17, 16, 24, 3, 2, 1, 1, "f32", 0.6),     # smaller still: fp32 gather convolution, stride 2
    (1, 16, 16, 32, 32, 3, 1, 32, 4, "bf16", 0.7),   # depthwise
]


def test_static_step_matches_handle_step():
    for ci, (n, h, w, c_in, c_out, k, stride, groups, block, dtype, eps) in enumerate(CASES):
        frames = [syn.to_storage(f, dtype) for f in syn.RectVideo(h, w, c_in, 3, seed=700 + ci, batch=n,
                                                                       side_lo=3, side_hi=6)]
        wf = syn.he_weights(c_out, c_in // groups, k, seed=710 + ci)
        wdev = to_device(weight_storage(wf, dtype), dtype)
        layer = S.SkipConv(wdev, n=n, h=h, w=w, stride=stride, groups=groups, eps=eps, block=block,
                           split=True, caller_retains=True)
        d = S.make_desc(n=n, h=h, w=w, c_in=c_in, c_out=c_out, kernel=k, stride=stride, groups=groups,
                        block=block, dtype=dtype, eps=eps)
        z = torch.full((n, layer.h_out, layer.w_out, c_out), float("nan"), dtype=torch.float32, device="cuda")
        stream = torch.cuda.current_stream().cuda_stream
        xs = [to_device(f, dtype) for f in frames]
        for t, x in enumerate(xs):
            say(f"[static] case {ci} frame {t}: n={n} {h}x{w} {c_in}->{c_out} k={k} s={stride} g={groups} "
                f"b={block} {dtype}")
            zh = layer.step(x)
            S.skipconv_step_static(d, wdev.data_ptr(), x.data_ptr(), xs[t - 1].data_ptr() if t else None,
                                   z.data_ptr(), stream)
            torch.cuda.synchronize()
            a, b = z.cpu().numpy(), zh.cpu().numpy()
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), f"case {ci} t={t}: z differs"
        blocks, _ = layer.active_count()
        say(f"[static] case {ci}: {blocks} active blocks on the last frame")
        layer.close()


def test_static_step_rejects_what_does_not_fit():
    # the work list of a per-site gate on 4 x 512 x 512 outputs needs more than the fixed scratch
    d = S.make_desc(n=4, h=512, w=512, c_in=128, c_out=128, kernel=3, block=1, dtype="bf16", eps=1.0)
    with pytest.raises(S.SkipConvError) as ei:
        S.skipconv_step_static(d, 16, 16, None, 16, 0)
    assert ei.value.code == S.SKIPCONV_E_SMALL_BUFFER
    assert "scratch" in S.skipconv_last_error(None)
    d = S.make_desc(n=1, h=16, w=16, c_in=32, c_out=32, kernel=3, block=8, dtype="bf16", eps=1.0,
                    keep_stats=True)
    with pytest.raises(S.SkipConvError) as ei:
        S.skipconv_step_static(d, 16, 16, None, 16, 0)
    assert ei.value.code == S.SKIPCONV_E_UNSUPPORTED
