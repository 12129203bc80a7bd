"""GPU test of the two read probes (the measurement aids behind
`bench.py --op read_ceiling`): it must read every 16-byte word exactly once,
which the xor of its per-wave sink words shows."""
import sys

import numpy as np
import pytest

import paper_2411_01142_amd as neo

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    neo.load_library()
    yield


# Sizes below one word per thread, with a partial last round, and several
# rounds of 8 loads per thread (the grid has 2^20 threads).
@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (1 << 24) + 16 * 7, 1 << 27])
@pytest.mark.parametrize("nontemporal", [False, True])
def test_read_probe_reads_every_word_once(nbytes, nontemporal):
    print(f"[probe] bytes={nbytes} nontemporal={nontemporal}", flush=True)
    sys.stdout.flush()
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 2 ** 32, nbytes // 4, dtype=np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.full((neo.READ_PROBE_SINK_WORDS,), -1, dtype=torch.int32, device="cuda")
    neo.read_probe(src, sink, nontemporal=nontemporal)
    torch.cuda.synchronize()
    words = sink.cpu().numpy().view(np.uint32)
    assert np.all(words != 0xFFFFFFFF)  # every wave wrote its word
    assert np.bitwise_xor.reduce(words) == np.bitwise_xor.reduce(host)


def test_read_probe_binding_checks():
    src = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError):
        neo.read_probe(src, torch.zeros(8, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError):
        neo.read_probe(src.cpu(), torch.zeros(neo.READ_PROBE_SINK_WORDS, dtype=torch.int32))


# One step (most waves empty), a count that leaves waves with unequal ranges,
# and several rounds of every depth's ring.
# With XCD weights the ranges follow the decode kernel's weighted slice
# geometry (too few steps per wave for it: equal ranges again).
@pytest.mark.parametrize("nbytes", [8192, 8192 * 1237, 1 << 27])
@pytest.mark.parametrize("wpc,depth", [(4, 1), (8, 2), (12, 3), (8, 4), (16, 1)])
@pytest.mark.parametrize("weighted", [False, True])
def test_tile_probe_reads_every_word_once(nbytes, wpc, depth, weighted):
    print(f"[probe-tiles] bytes={nbytes} waves/CU={wpc} depth={depth} xcd_weighted={weighted}",
          flush=True)
    sys.stdout.flush()
    rng = np.random.default_rng(nbytes + wpc + depth)
    host = rng.integers(0, 2 ** 32, nbytes // 4, dtype=np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(neo.READ_PROBE_SINK_WORDS, dtype=torch.int32, device="cuda")
    neo.read_probe_tiles(src, sink, waves_per_cu=wpc, depth=depth, xcd_weighted=weighted)
    torch.cuda.synchronize()
    words = sink.cpu().numpy().view(np.uint32)
    assert np.bitwise_xor.reduce(words) == np.bitwise_xor.reduce(host)


def test_tile_probe_rejects_bad_arguments():
    src = torch.zeros(4096, dtype=torch.int32, device="cuda")   # 16 KiB
    sink = torch.zeros(neo.READ_PROBE_SINK_WORDS, dtype=torch.int32, device="cuda")
    for kw in (dict(waves_per_cu=6), dict(waves_per_cu=20), dict(depth=0), dict(depth=5)):
        with pytest.raises(neo.NeoError):
            neo.read_probe_tiles(src, sink, **kw)
    with pytest.raises(neo.NeoError):
        neo.read_probe_tiles(src[:100], sink)                  # not a multiple of 8192 bytes
    with pytest.raises(neo.NeoError):
        neo.read_probe_tiles(src, sink[:16])                   # sink too small
