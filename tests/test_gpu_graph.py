"""The step as a HIP graph: rikfad_step only enqueues kernel launches on the
caller's stream (no allocation, no memset, no host synchronisation), so it
can be captured once and replayed -- the way to remove launch overhead for
small parameter sets, whose steps are launch-bound.  Every replay must give
the same bits as an eager twin driven with the same inputs, with eager work
and synchronisations between the replays."""
import pytest
import torch

from paper_2609_30342_amd import synth

from parity import load_grads, log, make_pair

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

S = synth.TensorSpec


@pytest.mark.parametrize("two_pass", [False, True])
def test_graph_replays_match_eager_bitwise(two_pass):
    # f: 66 row stripes (column items of 4 stripe lanes x 64 columns)
    specs = [S("a", 256, 512), S("b", 1, 512), S("c", 300, 27), S("d", 40, 640, "bf16"),
             S("e", 640, 1, "bf16"), S("f", 4200, 96)]
    hp = synth.HP_FRICTION
    log(f"[case] graph capture two_pass={two_pass}")
    eager = make_pair(specs, hp, seed=21, two_pass=two_pass, checked=[])
    graph = make_pair(specs, hp, seed=21, two_pass=two_pass, checked=[])
    # Warm-up step outside the capture (builds the factor sums, arms the
    # deferred half-kick).
    for pr in (eager, graph):
        load_grads(pr, 0, 21)
        pr.opt.step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graph.opt.step()
    torch.cuda.synchronize()
    for step in range(1, 7):
        load_grads(eager, step, 21)
        load_grads(graph, step, 21)
        eager.opt.step()
        g.replay()
        torch.cuda.synchronize()
        for i in range(len(specs)):
            assert torch.equal(eager.xs[i], graph.xs[i]), (step, i)
            for u, v in zip(eager.opt.state[i], graph.opt.state[i]):
                assert torch.equal(u, v), (step, i)
    eager.opt.sync_momentum()
    graph.opt.sync_momentum()
    torch.cuda.synchronize()
    for i in range(len(specs)):
        for u, v in zip(eager.opt.state[i], graph.opt.state[i]):
            assert torch.equal(u, v)


@pytest.mark.parametrize("name", ["gpt2_nano", "tinyvit"])
def test_graph_replays_match_oracle(name):
    """The launch-bound model-shaped sets stepped by replaying one captured
    step, checked against the fp64 oracle (not only against eager HIP):
    GPT2-Nano-shaped fp32 and TinyViT-shaped bf16, friction active, with a
    synchronisation and new gradients between the replays."""
    from parity import assert_ok, compare, oracle_step, reset_bf16_x
    specs = synth.gpt2_nano() if name == "gpt2_nano" else synth.tinyvit_like()
    hp = synth.HP_FRICTION
    log(f"[case] graph replay vs oracle {name} tensors={len(specs)}")
    pair = make_pair(specs, hp, seed=23)
    has_bf16 = any(o.bf16 for o in pair.ref.values())
    worst = 0.0

    def one(step, run):
        nonlocal worst
        if has_bf16:
            reset_bf16_x(pair)
        hg = load_grads(pair, step, 23)
        run()
        oracle_step(pair, hg, hp)
        if has_bf16:
            worst = max(worst, compare(pair, sync=False, what=("x",))["x_bf16"])

    one(0, pair.opt.step)              # eager first step: arms the deferred half-kick
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pair.opt.step()
    # the capture enqueued nothing: the graph's first replay is step 1
    for step in range(1, 9):
        one(step, g.replay)
        torch.cuda.synchronize()
    errs = compare(pair)
    if has_bf16:
        errs["x_bf16"] = max(errs["x_bf16"], worst)
    log(f"[graph] {name} errs={ {k: f'{v:.2e}' for k, v in errs.items()} }")
    assert_ok(errs, label=f"graph {name}")
