"""The Python binding refuses tensors the raw-pointer ABI cannot check: outputs
of the wrong shape, host tensors, non-contiguous views and wrong dtypes raise
before anything is launched."""
import numpy as np
import pytest

from paper_2607_07740_amd import api, synth
from parity_util import say, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _inputs(B=1, Hq=4, Hkv=2, L=130):
    return [to_dev(x) for x in synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=3)]


def test_prefill_output_shapes_are_checked():
    q, k, v = _inputs()
    say("binding checks: prefill outputs")
    short = torch.empty((1, 129, 4, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="out must have shape"):
        api.bifocal_prefill(q, k, v, w_pretrained=64, w_local=8, out=short)
    bad_lse = torch.empty((1, 130, 4), dtype=torch.float32, device="cuda")  # [B, L, Hq]
    with pytest.raises(ValueError, match="lse must have shape"):
        api.bifocal_prefill(q, k, v, w_pretrained=64, w_local=8, lse=bad_lse)
    with pytest.raises(ValueError, match="out must have shape"):
        api.prefill_chunk(q[:, 100:].contiguous(), k, v, q_start=100, w_pretrained=64, w_local=8,
                          out=torch.empty_like(q))
    with pytest.raises(ValueError, match="out must have shape"):
        api.bifocal_prefill_literal(q, k, v, w_pretrained=64, w_local=8, out=short)


def test_decode_output_shapes_are_checked():
    B, Hq, Hkv, max_len = 2, 4, 2, 300
    q, kc, vc, lens = synth.decode_inputs(B, Hq, Hkv, max_len, [300, 17], seed=4)
    qd, kd, vd = to_dev(q), to_dev(kc), to_dev(vc)
    ld = torch.from_numpy(lens).cuda()
    say("binding checks: decode outputs")
    wrong = torch.empty((B, Hq, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError, match="out must have shape"):
        api.bifocal_decode(qd, kd, vd, ld, w_pretrained=64, w_local=8, out=wrong)
    with pytest.raises(ValueError, match="out must have shape"):
        api.bifocal_decode(qd, kd, vd, ld, w_pretrained=64, w_local=8, out=wrong,
                           remote_map="freq")
    with pytest.raises(ValueError, match="out must have shape"):
        api.bifocal_decode_noalloc(qd, kd, vd, ld, w_pretrained=64, w_local=8, out=wrong)


def test_host_noncontiguous_and_mistyped_tensors_are_refused():
    q, k, v = _inputs()
    say("binding checks: inputs")
    with pytest.raises(TypeError, match="CUDA"):
        api.bifocal_prefill(q, k.cpu(), v, w_pretrained=64, w_local=8)
    with pytest.raises(ValueError, match="contiguous"):
        api.bifocal_prefill(q.transpose(1, 2).contiguous().transpose(1, 2), k, v,
                            w_pretrained=64, w_local=8)
    with pytest.raises(TypeError, match="bfloat16"):
        api.bifocal_prefill(q.float(), k, v, w_pretrained=64, w_local=8)
    # nothing above reached the device: a valid call still works and is finite
    out = api.bifocal_prefill(q, k, v, w_pretrained=64, w_local=8)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out.float()).all())
    assert np.isfinite(out.float().cpu().numpy()).all()
