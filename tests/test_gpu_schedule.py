"""The level-1 start (sd_start_level = 1): atspeed_decode_topk takes level 1
from the prefill's root log-probs and speculates from t = 1.  Strict
verification is lossless either way, so the lists, scores and counts must be
bitwise those of the Algorithm 1 schedule (t = 0), and the first step must
report zero accepted levels and t = 1 for every user."""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from _gpu_common import env  # noqa: E402

DEV = "cuda:0"


def _decode(eng, w, prefix, stats=None):
    items = torch.zeros((w.batch, w.K, w.L), dtype=torch.int32, device=DEV)
    scores = torch.zeros((w.batch, w.K), dtype=torch.float32, device=DEV)
    n = torch.zeros(w.batch, dtype=torch.int32, device=DEV)
    eng.atspeed_decode_topk(prefix, items, scores, n, stats)
    torch.cuda.synchronize()
    return items.cpu().numpy(), scores.cpu().numpy(), n.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_level_one_start_is_lossless(name):
    from paper_2410_05165_amd.binding import Engine, Stats
    e = env(name)
    w = e["w"]
    prefix = torch.from_numpy(e["pre"]).to(DEV)
    eng0 = Engine(w, e["tw"], e["dw"], e["cat"], sd_start_level=0)
    eng1 = Engine(w, e["tw"], e["dw"], e["cat"], sd_start_level=1)
    try:
        print(f"[{name}] decode with sd_start_level 0 and 1", flush=True)
        ref = _decode(eng0, w, prefix)
        acc = np.full((w.L, w.batch), -9, np.int32)
        ta = np.full((w.L, w.batch), -9, np.int32)
        st = Stats()
        st.accepted = acc.ctypes.data_as(C.POINTER(C.c_int32))
        st.t_after = ta.ctypes.data_as(C.POINTER(C.c_int32))
        got = _decode(eng1, w, prefix, st)
        print(f"[{name}] steps {st.n_steps}, t after each step {ta[:st.n_steps, :4].tolist()}")
        for x, y in zip(got, ref):
            np.testing.assert_array_equal(x, y)
        assert (acc[0] == 0).all() and (ta[0] == 1).all()
        assert 1 <= st.n_steps <= w.L
    finally:
        eng1.close()
        eng0.close()
