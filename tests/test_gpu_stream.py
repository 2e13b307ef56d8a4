"""GPU parity of the layer stream (one persistent launch for a sequence of
layers; the decode setting of Sec. 5.4) against the fp64 oracle.

Each item is checked element-wise against the oracle evaluated on the input
that item actually read: the caller's x, or (chained items) the GPU output
of an earlier item, so every layer of a chain is held to the single-layer
bar.  Outputs are prefilled with NaN, so a row a phase failed to write
cannot pass."""
import numpy as np
import pytest
import torch

from paper_2609_06161_amd import af1, synth
from paper_2609_06161_amd.layer import DeviceLayer, LayerStream, bf16_bits_to_f64, to_device

pytestmark = pytest.mark.gpu

TOL = 5e-3


def max_row_rel_l2(y, ref):
    worst = 0.0
    for a, e in zip(np.asarray(y, np.float64), np.asarray(ref, np.float64)):
        ne = np.linalg.norm(e)
        worst = max(worst, np.linalg.norm(a - e) / ne if ne > 0 else float(np.abs(a).max()))
    return worst


def elementwise_ok(y, ref, rel=2 ** -7, abs_rms=1e-3):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    bad = ~(np.abs(y - ref) <= rel * np.abs(ref) + abs_rms * scale)
    return not bad.any(), np.argwhere(bad)[:5]


def host_bits(t):
    return t.detach().cpu().numpy().view(np.uint16)


def nan_out(b, m):
    return torch.full((b, m), 0x7FC0, dtype=torch.int16, device="cuda")


def check_items(oracle, lins, entries):
    """entries: (DeviceLayer, x, y, wait); lins: the host layers."""
    for k, ((L, x, y, _), lin) in enumerate(zip(entries, lins)):
        xin = host_bits(x)
        ref = oracle.forward(lin.m, lin.n, lin.r, lin.Bu, lin.Bv, lin.s_out, lin.s_mid,
                             lin.s_in, xin)
        got = bf16_bits_to_f64(y)
        assert np.all(np.isfinite(ref))
        err = max_row_rel_l2(got, ref)
        ok, where = elementwise_ok(got, ref)
        assert err <= TOL and ok, (k, lin.m, lin.n, lin.r, err, where)


DECODER = [("q", 4096, 4096, 2016), ("k", 1024, 4096, 800), ("v", 1024, 4096, 800),
           ("o", 4096, 4096, 2016), ("gate", 14336, 4096, 3136),
           ("up", 14336, 4096, 3136), ("down", 4096, 14336, 3136)]


def decoder_entries(layers, b, seed, ranks=None):
    """A chained decoder: q/k/v read the block input; o reads q's output (in
    place of attention, same width) and waits; gate/up read o's output and
    wait; down reads gate's output (in place of the activation product) and
    waits; the next layer's q/k/v read down's output and wait."""
    lins, entries = [], []
    h = to_device(synth.make_activations(seed, b, 4096))
    for layer in range(layers):
        outs = {}
        for i, (name, m, n, r0) in enumerate(DECODER):
            r = ranks[7 * layer + i] if ranks is not None else r0
            lin = synth.make_linear(seed + 100 * layer + i, m, n, r, b)
            L = DeviceLayer.from_host(lin)
            x = {"q": h, "k": h, "v": h, "o": outs.get("q"), "gate": outs.get("o"),
                 "up": outs.get("o"), "down": outs.get("gate")}[name]
            wait = name in ("o", "gate", "down") or (name == "q" and layer > 0)
            y = nan_out(b, m)
            outs[name] = y
            lins.append(lin)
            entries.append((L, x, y, wait))
        h = outs["down"]
    return lins, entries


@pytest.mark.parametrize("b", [1, 4])
def test_stream_chained_decoder_layers(oracle, b):
    """Two 8B-shaped decoder layers (14 linears) with real data chaining and
    the stack's heterogeneous ranks."""
    linears = [(nm, m, n, r) for nm, m, n, r in DECODER]
    ranks = [e[4] for e in synth.draw_stack_ranks(77, 32, linears, af1.af1_storage_bits)][:14]
    print(f"stream decoder 2 layers b={b}", flush=True)
    lins, entries = decoder_entries(2, b, 9000 + b, ranks)
    S = LayerStream(entries, b)
    S.run()
    torch.cuda.synchronize()
    assert S.error_word() == 0
    check_items(oracle, lins, entries)


@pytest.mark.parametrize("b", [1, 8])
def test_stream_chain_of_square_layers(oracle, b):
    """Six 4096x4096 r=2016 layers, each reading the previous one's output."""
    print(f"stream 4096^2 chain b={b}", flush=True)
    x = to_device(synth.make_activations(9100 + b, b, 4096))
    lins, entries = [], []
    for i in range(6):
        lin = synth.make_linear(9110 + i, 4096, 4096, 2016, b)
        y = nan_out(b, 4096)
        entries.append((DeviceLayer.from_host(lin), x, y, i > 0))
        lins.append(lin)
        x = y
    S = LayerStream(entries, b)
    S.run()
    torch.cuda.synchronize()
    check_items(oracle, lins, entries)


@pytest.mark.parametrize("b", [1, 3, 16])
def test_stream_independent_and_ragged_items(oracle, b):
    """Items that do not wait (more than one group's worth, so a group's first
    product shares a phase with the previous group's second), ragged shapes
    with odd word counts, and, at b = 16, column slabs added by the last
    slab of a row group."""
    shapes = [(96, 2080, 160), (544, 4128, 96), (1056, 2080, 4064), (32, 32, 32),
              (4128, 14336, 3136), (1056, 64, 2080), (96, 1056, 96), (4096, 4096, 2016),
              (14368, 4096, 3136), (64, 96, 64)]
    print(f"stream independent items b={b}", flush=True)
    lins, entries = [], []
    for i, (m, n, r) in enumerate(shapes):
        lin = synth.make_linear(9200 + 10 * b + i, m, n, r, b)
        entries.append((DeviceLayer.from_host(lin), to_device(lin.x), nan_out(b, m), False))
        lins.append(lin)
    S = LayerStream(entries, b)
    S.run()
    torch.cuda.synchronize()
    check_items(oracle, lins, entries)


def test_stream_repeated_passes_and_graph_replay(oracle):
    """Five passes on one workspace (the arrival epoch advances every pass),
    then the pass captured in a HIP graph and replayed three times with
    eager work in between: every pass gives the same bits."""
    lins, entries = decoder_entries(1, 2, 9300)
    S = LayerStream(entries, 2)
    S.run()
    torch.cuda.synchronize()
    check_items(oracle, lins, entries)
    ref = [e[2].clone() for e in entries]
    for _ in range(4):
        for e in entries:
            e[2].fill_(0x7FC0)
        S.run()
        torch.cuda.synchronize()
        assert all(torch.equal(e[2], r) for e, r in zip(entries, ref))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        S.run()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        S.run()
    for _ in range(3):
        for e in entries:
            e[2].fill_(0x7FC0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert all(torch.equal(e[2], r) for e, r in zip(entries, ref))
    assert S.error_word() == 0


def test_stream_matches_single_calls_bitwise():
    """A stream item's output is what af1_linear_gemv gives for the layer
    (same kernels and plans at b = 1 for a layer alone in its phase)."""
    lin = synth.make_linear(9400, 4096, 4096, 2016, 1)
    L = DeviceLayer.from_host(lin)
    x = to_device(lin.x)
    y = nan_out(1, 4096)
    S = LayerStream([(L, x, y, False)], 1)
    S.run()
    y1 = L.gemv(x)
    torch.cuda.synchronize()
    assert torch.equal(y, y1)
