"""Pins of the oracle's whitespace proxy (stage 1) against Python itself.

The paper counts input words with str.split() under Python 3.10
(Sec. "Workload Characterization and Token Budget Estimation", and the
software table of Sec. "Experimental Hardware and Software Environment").
The running interpreter is therefore the reference: its str.isspace() set,
its str.split() and its UTF-8 decoder with the surrogateescape handler.
"""
import random

import numpy as np
import pytest

from tests import wl


def _pack(prompts):
    """bytes prompts -> (text uint8, offsets uint64)."""
    lens = [len(p) for p in prompts]
    offsets = np.zeros(len(prompts) + 1, dtype=np.uint64)
    offsets[1:] = np.cumsum(lens, dtype=np.uint64)
    text = np.frombuffer(b"".join(prompts), dtype=np.uint8).copy()
    return text, offsets


def _py_count(b):
    return len(b.decode("utf-8", "surrogateescape").split())


def test_space_table_matches_python(oracle):
    # every code point: the oracle's table == str.isspace()
    lib = oracle._load()
    mismatches = [cp for cp in range(0x110000) if bool(lib.dsref_is_space(cp)) != chr(cp).isspace()]
    assert mismatches == []
    assert sum(chr(cp).isspace() for cp in range(0x110000)) == 29


def test_split_separators_are_isspace_set(oracle):
    # str.split() separates on exactly the isspace() set; checked through the
    # oracle on "a<cp>b" for every encodable code point
    cps = [cp for cp in range(0x110000) if not (0xD800 <= cp <= 0xDFFF)]
    prompts = [("a" + chr(cp) + "b").encode("utf-8") for cp in cps]
    text, offsets = _pack(prompts)
    got = oracle.characterize(text, offsets)
    want = np.array([len(("a" + chr(cp) + "b").split()) for cp in cps], dtype=np.uint32)
    assert np.array_equal(got, want)
    assert int((want == 2).sum()) == 29


HAND = [
    (b"", 0),
    (b" ", 0),
    (b" \t\n\r\x0b\x0c\x1c\x1d\x1e\x1f", 0),
    (b"word", 1),
    (b"  two words  ", 2),
    (b"a\tb\nc\rd", 4),
    (b"a\x00b", 1),                         # NUL is not whitespace
    (b"a\x08b\x0eb", 1),                    # neither are other C0 controls
    ("a\u00a0b".encode(), 2),               # C2 A0 no-break space
    ("a\u0085b".encode(), 2),               # C2 85 next line
    ("a\u1680b".encode(), 2),               # E1 9A 80 ogham space mark
    ("a\u2000b\u200ac".encode(), 3),        # E2 80 80 and E2 80 8A
    ("a\u2028b\u2029c\u202fd\u205fe\u3000f".encode(), 6),
    ("\u00c5\u00e0".encode(), 1),           # C3 85 / C3 A0: letters, not spaces
    ("x\u2010y".encode(), 1),               # E2 80 90 hyphen
    ("x\u200by".encode(), 1),               # zero width space is not whitespace
    ("\u3007\u3000\u3007".encode(), 2),     # E3 80 87 is a letter, E3 80 80 a space
    (b"\xc2", 1),                           # truncated sequence: one character
    (b"a\xc2 b", 2),
    (b"\xe2\x80", 1),                       # truncated E2 80
    (b"a\xe2\x80\x41b", 1),                 # E2 80 then 'A': invalid, no space
    (b"\xe2\xe2\x80\x80x", 2),              # invalid E2, then U+2000, then x
    (b"\xed\xa0\x80 a", 2),                 # encoded surrogate is ill-formed
    (b"\xf0\x9f\x98\x80 \xf0\x9f", 2),
]


@pytest.mark.parametrize("raw,want", HAND)
def test_hand_cases(oracle, raw, want):
    assert _py_count(raw) == want          # the hand value is Python's
    assert oracle.count_words(raw) == want


def test_adjacent_prompts_do_not_merge(oracle):
    text, offsets = _pack([b"ab", b"cd", b"", b"e ", b" f", "\u3000".encode()])
    assert list(oracle.characterize(text, offsets)) == [1, 1, 0, 1, 1, 0]


def test_split_sequence_across_prompts(oracle):
    # a whitespace sequence cut by a prompt boundary is ill-formed in both
    # halves: each prompt is decoded on its own
    ws = "\u3000".encode()                   # E3 80 80
    prompts = [b"a" + ws[:2], ws[2:] + b"b", b"a" + ws[:1], ws[1:] + b"b"]
    text, offsets = _pack(prompts)
    got = oracle.characterize(text, offsets)
    assert list(got) == [_py_count(p) for p in prompts] == [1, 1, 1, 1]


ALPHABET = (
    [chr(cp) for cp in range(0x110000) if chr(cp).isspace()]
    + list("abcxyz019.,;")
    + ["\u00c5", "\u00e0", "\u00b5", "\u0420", "\u2c65", "\u3042", "\u4e00",
       "\u2010", "\u200b", "\u3007", "\u1e00", "\u00a9"]
    + ["\x00", "\x01", "\x07", "\x08", "\x0e", "\x1b", "\x7f"]
)


def test_fuzz_valid_utf8(oracle):
    rng = random.Random(12345)
    prompts = []
    for _ in range(100000):
        k = rng.randint(0, 24)
        prompts.append("".join(rng.choice(ALPHABET) for _ in range(k)).encode("utf-8"))
    text, offsets = _pack(prompts)
    got = oracle.characterize(text, offsets)
    want = np.array([len(p.decode("utf-8").split()) for p in prompts], dtype=np.uint32)
    assert np.array_equal(got, want)


def test_fuzz_arbitrary_bytes(oracle):
    # malformed input: the count equals Python's on the surrogateescape decode
    rng = random.Random(777)
    pieces = [b"\xc2", b"\x85", b"\xa0", b"\xe1", b"\x9a", b"\x80", b"\xe2", b"\x81",
              b"\x9f", b"\xa8", b"\xe3", b"\xed", b"\xf0", b"\xbf", b"a", b" ", b"\t"]
    prompts = []
    for _ in range(50000):
        k = rng.randint(0, 16)
        prompts.append(b"".join(rng.choice(pieces) for _ in range(k)))
    text, offsets = _pack(prompts)
    got = oracle.characterize(text, offsets)
    want = np.array([_py_count(p) for p in prompts], dtype=np.uint32)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("name,n", [("batch4k", None), ("long16k", 64)])
def test_generator_word_counts(oracle, name, n):
    # the generator records how many words it wrote into each prompt
    b = wl.load(name, n=n)
    got = oracle.characterize(b.text, b.offsets)
    assert np.array_equal(got, b.words)


def test_rejects_bad_offsets(oracle):
    with pytest.raises(ValueError):
        oracle.characterize(np.zeros(4, np.uint8), np.array([0, 3, 2], np.uint64))
    with pytest.raises(ValueError):
        oracle.characterize(np.zeros(4, np.uint8), np.array([0, 5], np.uint64))
