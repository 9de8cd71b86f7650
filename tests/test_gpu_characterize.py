"""Stage 1 on the GPU against the oracle: exact integer counts.

Covers hand cases, multi-byte separators at every alignment and across
chunk, round and wave boundaries, tiny and empty prompts (many boundaries
per round), bytes outside every prompt, ragged buffer tails, the five
workloads' text at full size, determinism and the DS_VALIDATE path.
"""
import random

import numpy as np
import pytest

import workloads as synth
from tests import wl
from tests.gpu_util import dev, host, pack

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def run(ds, text, offsets):
    c = ds.characterize(dev(text), dev(offsets))
    return host(c, np.uint32)


def check(ds, oracle, text, offsets):
    want = oracle.characterize(text, offsets)
    got = run(ds, text, offsets)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, "prompt %d: got %d want %d (of %d mismatches)" % (
        bad[0], got[bad[0]], want[bad[0]], bad.size)
    return got


SPACES = [chr(cp) for cp in range(0x110000) if chr(cp).isspace()]
LOOKALIKES = ["\u00c5", "\u00e0", "\u00b5", "\u0420", "\u2c65", "\u3042", "\u4e00", "\u2010",
              "\u200b", "\u3007", "\u1e00", "\u00a9", "\u2030", "\u205e", "\u3001", "\u1681"]


def test_hand_cases(ds, oracle):
    from tests.test_oracle_characterize import HAND
    prompts = [raw for raw, _ in HAND]
    text, offsets = pack(prompts)
    got = check(ds, oracle, text, offsets)
    assert list(got) == [want for _, want in HAND]


def test_single_prompt_sizes(ds, oracle):
    # one prompt of every length 0..300 and around the 16/1024 byte steps
    rng = random.Random(3)
    alpha = SPACES + list("abcdefgh") + LOOKALIKES
    for L in list(range(0, 70)) + [1023, 1024, 1025, 4095, 4096, 4097, 20000]:
        s = "".join(rng.choice(alpha) for _ in range(L)).encode()
        text, offsets = pack([s])
        check(ds, oracle, text, offsets)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_fuzz_dense_multibyte(ds, oracle, seed):
    # ~2 MB of text dense in multi-byte separators and look-alikes, cut into
    # prompts of random lengths: separators land on every 16-byte alignment
    # and across round and wave-range boundaries
    rng = random.Random(seed)
    alpha = SPACES * 3 + list("abcdefghij") * 4 + LOOKALIKES * 2 + ["\x00", "\x1b", "\x7f"]
    prompts = []
    total = 0
    while total < 2_000_000:
        L = rng.choice([0, 1, 2, 3, 5, 17, 40, 300, 1500, 9000])
        s = "".join(rng.choice(alpha) for _ in range(L)).encode()
        prompts.append(s)
        total += len(s)
    text, offsets = pack(prompts)
    check(ds, oracle, text, offsets)


def test_fuzz_arbitrary_bytes(ds, oracle):
    rng = np.random.default_rng(11)
    pieces = [b"\xc2", b"\x85", b"\xa0", b"\xe1", b"\x9a", b"\x80", b"\xe2", b"\x81", b"\x9f",
              b"\xa8", b"\xe3", b"\xed", b"\xf0", b"\xbf", b"a", b" ", b"\t", b"b", b"\n"]
    idx = rng.integers(0, len(pieces), 1_500_000)
    blob = b"".join(pieces[i] for i in idx)
    cuts = np.sort(rng.integers(0, len(blob), 60000))
    bounds = np.concatenate(([0], cuts, [len(blob)]))
    prompts = [blob[bounds[i]:bounds[i + 1]] for i in range(len(bounds) - 1)]
    text, offsets = pack(prompts)
    check(ds, oracle, text, offsets)


def test_tiny_and_empty_prompts(ds, oracle):
    # thousands of prompt boundaries inside one 1 KiB round, runs of empty
    # prompts at the same position
    rng = np.random.default_rng(5)
    prompts = []
    for _ in range(60000):
        k = int(rng.integers(0, 4))
        prompts.append(bytes(rng.choice(list(b"ab \t\n"), size=k).tolist()) if k else b"")
    prompts += [b""] * 500 + [b"x"] * 3000 + [b""] * 70 + [b" "] * 200
    text, offsets = pack(prompts)
    check(ds, oracle, text, offsets)


def test_bytes_outside_prompts_and_ragged_tail(ds, oracle):
    rng = np.random.default_rng(6)
    body = synth.make_text(rng.integers(1, 300, 500).astype(np.uint32), 9, 0.05)
    text, offsets = body
    # prompts cover only a middle part; bytes before and after are ignored
    n = len(offsets) - 1
    for lo, hi in [(0, n), (3, n), (0, n - 5), (7, n - 9)]:
        off = offsets[lo:hi + 1].copy()
        check(ds, oracle, text, off)
    # buffer lengths that are not multiples of 16
    for cut in [1, 5, 15, 17, 1000, 4097]:
        t = text[:cut].copy()
        off = np.array([0, cut], dtype=np.uint64)
        check(ds, oracle, t, off)


def test_separator_split_by_prompt_boundary(ds, oracle):
    ws = "\u3000".encode()
    prompts = []
    for _ in range(200):
        prompts += [b"a" + ws[:2], ws[2:] + b"b", b"a" + ws[:1], ws[1:] + b"b", b"c\xc2", b"\xa0d"]
    text, offsets = pack(prompts)
    got = check(ds, oracle, text, offsets)
    assert set(got.tolist()) == {1}


def test_empty_text(ds, oracle):
    text = np.zeros(0, np.uint8)
    offsets = np.zeros(5, np.uint64)
    got = run(ds, text, offsets)
    assert list(got) == [0, 0, 0, 0]


@pytest.mark.parametrize("name", ["batch4k", "batch64k", "chat1m", "long16k"])
def test_workloads_full_size(ds, oracle, name):
    b = wl.load(name)
    got = check(ds, oracle, b.text, b.offsets)
    assert np.array_equal(got, b.words)


def test_deterministic(ds):
    b = wl.load("batch4k")
    t, o = dev(b.text), dev(b.offsets)
    a1 = host(ds.characterize(t, o))
    a2 = host(ds.characterize(t, o))
    assert np.array_equal(a1, a2)


def test_validate_flag(ds):
    text = dev(np.frombuffer(b"ab cd ef", np.uint8).copy())
    good = dev(np.array([0, 2, 8], np.uint64))
    c = ds.characterize(text, good, validate=True)
    assert list(host(c)) == [1, 2]
    for bad in ([0, 5, 3], [0, 2, 9]):
        with pytest.raises(ds.DriftSchedError) as e:
            ds.characterize(text, dev(np.array(bad, np.uint64)), validate=True)
        assert e.value.status == -5


@pytest.mark.parametrize("density", [0.002, 0.01, 0.05])
def test_long_prompts_sparse_multibyte(ds, oracle, density):
    # long prompts (no prompt boundary for many KiB) of ASCII words with
    # multi-byte separators and look-alikes sprinkled at every byte offset,
    # including across 1 KiB rounds and 4 KiB super-rounds
    rng = random.Random(int(density * 1000))
    seps = [c for c in SPACES if len(c.encode()) > 1]
    prompts = []
    for _ in range(12):
        parts = []
        size = 0
        while size < 300_000:
            x = rng.random()
            if x < density:
                t = rng.choice(seps)
            elif x < 2 * density:
                t = rng.choice(LOOKALIKES)
            elif x < 0.15:
                t = " "
            else:
                t = rng.choice("abcdefghij")
            parts.append(t)
            size += len(t.encode())
        prompts.append("".join(parts).encode())
    text, offsets = pack(prompts)
    got = check(ds, oracle, text, offsets)
    want = np.array([len(p.decode().split()) for p in prompts], dtype=np.uint32)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("nbytes", [0, 16, 4096 + 16, (10 << 20) + 48, 64 << 20])
def test_read_bandwidth_xor(nbytes):
    # the measurement aid reads every byte: the XOR of the buffer's words
    from paper_2606_02982_amd import driftsched as ds
    rng = np.random.default_rng(nbytes)
    host_buf = rng.integers(0, 256, nbytes, dtype=np.uint8)
    print("read_bandwidth bytes=%d" % nbytes, flush=True)
    out = host(ds.read_bandwidth(dev(host_buf)), np.uint32)
    assert out.size == ds.READ_BW_WORDS
    want = np.bitwise_xor.reduce(host_buf.view(np.uint32)) if nbytes else np.uint32(0)
    assert np.bitwise_xor.reduce(out) == np.uint32(want)
