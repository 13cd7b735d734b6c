"""A whole step captured in a HIP graph replays to the eager result, replay
after replay, with eager work and synchronisation between the replays."""
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import synth  # noqa: E402
from paper_2109_12497_amd.step import RandKStep, Step, capture  # noqa: E402

DEV = torch.device("cuda:0")


@pytest.mark.parametrize("kind", ["single", "multi", "packed", "streamed", "randk"])
def test_graph_replays_match_eager(kind):
    d, M = 200_003, 4
    host = synth.mixed_rows(M, d, seed=17, ldg=synth.round_up(d, 64))
    g = torch.from_numpy(host).to(DEV)
    if kind == "single":
        st = Step(d, M, [127.0], device=DEV)
    elif kind == "multi":
        st = Step(d, M, synth.scales_for(8, 4), device=DEV)
    elif kind == "packed":
        st = Step(d, M, synth.scales_for(4, 2), device=DEV, bits=4)
    elif kind == "streamed":
        st = Step(d, M, synth.scales_for(8, 3), device=DEV, streamed=True)
    else:
        st = RandKStep(d, M, 5000, synth.scales_for(8, 2), device=DEV)
    st.run(g, seed=3)
    torch.cuda.synchronize()
    ref = st.out[:d].clone()
    graph = capture(st, g, seed=3)
    for _ in range(4):
        st.out.fill_(-1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(st.out[:d], ref)
        st.run(g, seed=4)  # different eager work between the replays
        torch.cuda.synchronize()
        assert not torch.equal(st.out[:d], ref)
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(st.out[:d], ref)
