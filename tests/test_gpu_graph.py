"""A whole decode step (mcd_head_step) captured once in a HIP graph and
replayed: the library allocates nothing, synchronises nothing and records no
memset, so a serving loop can capture its step.  Every replay, fed new hidden
states and step numbers through the captured buffers, must give the tokens,
scores and frame grid of the same step run eagerly on a twin workload."""
import numpy as np
import pytest

from paper_2607_02119_amd import inputs
from tests._compare import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2607_02119_amd import harness, mcd  # noqa: E402

CASES = [
    # streaming kernel, top-p
    ("graph_stream", dict(H=256, K=4, V=300, n_pairs=6, n_solo=2, dtype="bf16", top_p=0.9,
                          steps=8, shuffle=True)),
    # audio and text rows on two streams (fork and join inside the graph)
    ("graph_two_streams", dict(H=128, K=3, V=37, n_pairs=10, n_solo=5, n_text=3, V_text=300,
                               dtype="bf16", top_k=7, steps=6, shuffle=True)),
    # more than 128 audio rows below 256 tiles of 256 x 256: 128 x 256
    # streaming row tiles in the XCD-aware order (3 x 8 tiles)
    ("graph_row_tiles", dict(H=256, K=4, V=512, n_pairs=140, n_solo=20, dtype="bf16", top_k=20,
                             steps=6, shuffle=True)),
    # the single mixed launch (256 tiles of 256 x 256 and 70 text rows)
    ("graph_fused_mixed", dict(H=64, K=8, V=4093, n_pairs=100, n_solo=60, n_text=70,
                               V_text=900, dtype="bf16", top_k=15, steps=9, shuffle=True)),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_step_replayed_from_a_graph_equals_eager(name, kw):
    wl = inputs.Workload(name, **kw)
    say(f"case graph {name} R={wl.R} N={wl.N} text={wl.n_text}")
    eager = harness.DeviceWorkload(wl)
    eager.load_hidden()
    twin = harness.DeviceWorkload(wl)
    h = torch.empty_like(eager.hidden[0])
    st = torch.empty_like(eager.step_tab[0])
    kwargs = twin.step_kwargs(0, h)
    kwargs["step"] = st
    handle = twin.heads[0].handle
    h.copy_(eager.hidden[0])
    st.copy_(eager.step_tab[0])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        mcd.mcd_head_step(handle, stream=side, **kwargs)        # warm-up, eager
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    twin.grid.fill_(-1)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        mcd.mcd_head_step(handle, **kwargs)
    for t in range(wl.steps):
        h.copy_(eager.hidden[t])
        st.copy_(eager.step_tab[t])
        torch.cuda.synchronize()
        g.replay()
        eager.run_step(t)
        torch.cuda.synchronize()
        assert np.array_equal(twin.tokens.cpu().numpy(), eager.tokens.cpu().numpy()), t
        assert torch.equal(twin.scores, eager.scores), t
    assert np.array_equal(twin.grid.cpu().numpy(), eager.grid.cpu().numpy())
    assert eager.status() == 0 and twin.status() == 0
