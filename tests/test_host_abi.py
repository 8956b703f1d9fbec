"""Host-side parts of libhvd, checked without a GPU.

* The C ABI: every function include/hvd.h declares is exported by libhvd.so
  and bound by the Python binding (and nothing else is).
* The page allocator and verify/commit state machine of the KV handle
  (host_state.cpp, through the host-only build libhvd_host.so): the verify
  rows of a sequence are the pending token plus k drafts at positions
  ctx .. ctx + k (the Verify interface of section 3.1); commit appends the
  accepted block z_t = draft[0:keep] + one target token (Alg. 1), so the
  cached length grows by keep + 1; every check happens before any page moves.
* The device-resident loop's host side: its page reservation for the longest
  outcome, the lock on the looping sequences, and the hand-back at its end.
"""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_01019_amd")
HEADER = os.path.join(ROOT, "include", "hvd.h")

OK, ARG, STATE, OOM, RANGE = 0, -1, -2, -3, -4
PAGE = 16


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)  # comments mention calls too
    return set(re.findall(r"\b(hvd_\w+)\s*\(", text))


def test_header_functions_are_exported_and_bound():
    from paper_2606_01019_amd import hvd
    declared = header_functions()
    assert declared == set(hvd.EXPORTS), declared ^ set(hvd.EXPORTS)
    lib_path = os.path.join(PKG, "libhvd.so")
    if not os.path.exists(lib_path):
        pytest.skip("libhvd.so not built (python -m paper_2606_01019_amd.build)")
    out = subprocess.run(["nm", "-D", "--defined-only", lib_path], capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    missing = sorted(n for n in declared if n not in exported)
    assert not missing, missing
    lib = hvd.load_library()
    for name in declared:
        assert getattr(lib, name) is not None


# ---------------------------------------------------------------- host state

P = ctypes.POINTER(ctypes.c_int32)


@pytest.fixture(scope="module")
def hostlib(tmp_path_factory):
    path = os.path.join(PKG, "libhvd_host.so")
    csrc = os.path.join(PKG, "csrc")
    srcs = [os.path.join(csrc, f) for f in ("host_state.cpp", "host_capi.cpp")]
    if not os.path.exists(path) or any(os.path.getmtime(s) > os.path.getmtime(path) for s in srcs):
        path = str(tmp_path_factory.mktemp("hostlib") / "libhvd_host.so")
        subprocess.run(["g++", "-O1", "-std=c++17", "-fPIC", "-shared", *srcs, "-o", path], check=True)
    L = ctypes.CDLL(path)
    V = ctypes.c_void_p
    I = ctypes.c_int32
    sig = {
        "hvdh_create": (V, [I, I, I, I, I]),
        "hvdh_destroy": (None, [V]),
        "hvdh_prefill": (I, [V, I, P, I]),
        "hvdh_begin_verify": (I, [V, I, P, P, P, P]),
        "hvdh_finish_verify": (None, [V, I, P, P, P, P, P]),
        "hvdh_abort_verify": (None, [V, I, P]),
        "hvdh_commit": (I, [V, I, P, P]),
        "hvdh_begin_async": (I, [V, I, P, P, P, I]),
        "hvdh_end_async": (None, [V, I, P, P, P]),
        "hvdh_truncate": (I, [V, I, I, I]),
        "hvdh_free_seq": (I, [V, I]),
        "hvdh_free_pages": (I, [V]),
        "hvdh_seq": (I, [V, I, P]),
        "hvdh_pages": (I, [V, I, P, I]),
        "hvdh_error": (ctypes.c_char_p, [V]),
    }
    for n, (r, a) in sig.items():
        f = getattr(L, n)
        f.restype = r
        f.argtypes = a
    return L


def arr(xs):
    a = np.ascontiguousarray(np.asarray(xs, dtype=np.int32))
    return a, (a.ctypes.data_as(P) if a.size else None)


class Host:
    """Thin wrapper: one HostState with max_pos 4096, max_draft 64, vocab 1000."""

    def __init__(self, L, max_seqs=4, n_pages=64, max_pos=4096, max_draft=64, vocab=1000):
        self.L = L
        self.h = L.hvdh_create(max_seqs, n_pages, max_pos, max_draft, vocab)
        self.keep = []

    def _a(self, xs):
        a, p = arr(xs)
        self.keep.append(a)
        return p

    def prefill(self, sid, toks):
        return self.L.hvdh_prefill(self.h, sid, self._a(toks), len(toks))

    def verify(self, ids, ctx, drafts, acc=None, nxt=None):
        """begin_verify, then (on success) record accepted / next as the device would."""
        lens = [len(d) for d in drafts]
        flat = [t for d in drafts for t in d]
        st = self.L.hvdh_begin_verify(self.h, len(ids), self._a(ids), self._a(ctx), self._a(flat), self._a(lens))
        if st == OK and acc is not None:
            self.L.hvdh_finish_verify(self.h, len(ids), self._a(ids), self._a(flat), self._a(lens), self._a(acc),
                                      self._a(nxt))
        return st

    def commit(self, ids, keep=None):
        return self.L.hvdh_commit(self.h, len(ids), self._a(ids), self._a(keep) if keep is not None else None)

    def truncate(self, sid, ctx, pend):
        return self.L.hvdh_truncate(self.h, sid, ctx, pend)

    def begin_async(self, ids, ctx, lens, steps):
        return self.L.hvdh_begin_async(self.h, len(ids), self._a(ids), self._a(ctx), self._a(lens), steps)

    def end_async(self, ids, ctx, pend):
        self.L.hvdh_end_async(self.h, len(ids), self._a(ids), self._a(ctx), self._a(pend))

    def seq(self, sid):
        out, p = arr([0, 0, 0, 0])
        if self.L.hvdh_seq(self.h, sid, p) != 0:
            return None
        return dict(ctx=int(out[0]), pending=int(out[1]), verify_pending=bool(out[2]), pages=int(out[3]))

    def pages(self, sid):
        out, p = arr(np.zeros(512))
        n = self.L.hvdh_pages(self.h, sid, p, 512)
        return [int(x) for x in out[:n]]

    def free(self):
        return self.L.hvdh_free_pages(self.h)

    def error(self):
        return self.L.hvdh_error(self.h).decode()

    def close(self):
        self.L.hvdh_destroy(self.h)


def pages_for(n):
    return (n + PAGE - 1) // PAGE


@pytest.fixture
def host(hostlib):
    h = Host(hostlib)
    yield h
    h.close()


def test_prefill_holds_prompt_and_pending(host):
    assert host.prefill(0, list(range(1, 41))) == OK
    s = host.seq(0)
    assert s == dict(ctx=39, pending=40, verify_pending=False, pages=pages_for(40))
    assert host.free() == 64 - pages_for(40)
    assert host.prefill(0, [1, 2]) == ARG  # id in use
    assert host.prefill(1, []) == ARG
    assert host.prefill(1, [1, 1000]) == RANGE
    assert host.prefill(9, [1]) == ARG


def test_verify_commit_keeps_accepted_block_plus_one(host):
    host.prefill(0, list(range(1, 33)))  # ctx 31, pending 32
    draft = [5, 6, 7, 8, 9, 10, 11]
    assert host.verify([0], [31], [draft], acc=[4], nxt=[77]) == OK
    # pages for the pending row plus 7 drafts: positions 0 .. 38
    assert host.seq(0)["pages"] == pages_for(31 + 7 + 1) and host.seq(0)["verify_pending"]
    assert host.verify([0], [31], [draft]) == STATE  # not committed yet
    assert host.commit([0], keep=[5]) == ARG  # keep > accepted
    assert host.commit([0]) == OK  # keep = accepted = 4: 4 drafts + the target token
    assert host.seq(0) == dict(ctx=36, pending=77, verify_pending=False, pages=pages_for(37))
    assert host.commit([0]) == STATE  # commit without a verify


def test_commit_shorter_keep_takes_the_draft_token_as_pending(host):
    host.prefill(0, list(range(1, 11)))  # ctx 9
    assert host.verify([0], [9], [[21, 22, 23]], acc=[3], nxt=[99]) == OK
    assert host.commit([0], keep=[1]) == OK
    assert host.seq(0)["ctx"] == 11 and host.seq(0)["pending"] == 22
    assert host.verify([0], [11], [[]], acc=[0], nxt=[5]) == OK  # k = 0: plain greedy step
    assert host.commit([0], keep=[0]) == OK
    assert host.seq(0)["ctx"] == 12 and host.seq(0)["pending"] == 5


def test_verify_errors_take_no_pages(hostlib):
    h = Host(hostlib, n_pages=8, max_pos=200, max_draft=8)
    try:
        assert h.prefill(0, list(range(1, 17))) == OK  # 1 page
        assert h.prefill(1, list(range(1, 17))) == OK
        free0 = h.free()
        assert h.verify([0, 0], [15, 15], [[1], [2]]) == ARG  # duplicate
        assert h.verify([3], [0], [[1]]) == ARG  # unknown
        assert h.verify([0], [14], [[1]]) == STATE  # ctx disagrees
        assert h.verify([0], [15], [[1] * 9]) == RANGE  # k > max_draft
        assert h.verify([0], [15], [[1, 1000]]) == RANGE  # token outside the vocabulary
        # a failed device step gives the reserved pages back
        assert h.verify([0, 1], [15, 15], [[1] * 8, [1] * 8]) == OK
        assert h.free() == free0 - 2
        h.L.hvdh_abort_verify(h.h, 2, h._a([0, 1]))
        assert h.free() == free0
        big = Host(hostlib, n_pages=3, max_pos=200, max_draft=64)
        try:
            big.prefill(0, list(range(1, 17)))
            big.prefill(1, list(range(1, 17)))
            f = big.free()
            assert big.verify([0, 1], [15, 15], [[1] * 8, [1] * 30]) == OOM
            assert big.free() == f and big.seq(0)["pages"] == 1
        finally:
            big.close()
        # rotary table: positions ctx .. ctx + k must stay below max_pos
        h2 = Host(hostlib, n_pages=64, max_pos=40, max_draft=8)
        try:
            h2.prefill(0, list(range(1, 36)))  # ctx 34
            assert h2.verify([0], [34], [[1] * 6]) == RANGE  # position 40
            assert h2.verify([0], [34], [[1] * 5]) == OK  # positions up to 39
        finally:
            h2.close()
    finally:
        h.close()


def test_truncate_and_free_return_pages(host):
    host.prefill(0, list(range(1, 101)))  # ctx 99, 7 pages
    assert host.truncate(0, 40, 7) == OK
    assert host.seq(0) == dict(ctx=40, pending=7, verify_pending=False, pages=pages_for(41))
    assert host.truncate(0, 41, 7) == ARG
    assert host.L.hvdh_free_seq(host.h, 0) == OK
    assert host.free() == 64 and host.seq(0) is None


def test_async_loop_reserves_longest_outcome_and_locks(host):
    host.prefill(0, list(range(1, 51)))  # ctx 49
    host.prefill(1, list(range(1, 21)))  # ctx 19
    free0 = host.free()
    steps, k = 10, 8
    assert host.begin_async([0], [49], [k], steps) == OK
    # the loop can commit up to steps * (k + 1) tokens; the page of the final pending token is held too
    assert host.seq(0)["pages"] == pages_for(49 + steps * (k + 1) + 1)
    for call in (lambda: host.verify([0], [49], [[1]]), lambda: host.commit([0]),
                 lambda: host.truncate(0, 10, 1), lambda: host.L.hvdh_free_seq(host.h, 0),
                 lambda: host.begin_async([0], [49], [k], 1)):
        assert call() == STATE
        assert "device-resident" in host.error()
    # other sequences keep working
    assert host.verify([1], [19], [[3, 4]], acc=[2], nxt=[9]) == OK and host.commit([1]) == OK
    # the loop ends after committing 23 tokens: pages past the new pending position return
    host.end_async([0], [49 + 23], [555])
    assert host.seq(0) == dict(ctx=72, pending=555, verify_pending=False, pages=pages_for(73))
    assert host.free() == free0 - (pages_for(73) - pages_for(50)) - (pages_for(23) - pages_for(20))
    assert host.verify([0], [72], [[1]], acc=[1], nxt=[2]) == OK


def test_async_loop_checks_before_reserving(hostlib):
    h = Host(hostlib, n_pages=12, max_pos=300, max_draft=16)
    try:
        h.prefill(0, list(range(1, 17)))  # ctx 15, 1 page
        h.prefill(1, list(range(1, 17)))
        f = h.free()
        assert h.begin_async([0], [15], [4], 0) == ARG
        assert h.begin_async([0, 0], [15, 15], [4, 4], 2) == ARG
        assert h.begin_async([0], [14], [4], 2) == STATE
        assert h.begin_async([0], [15], [17], 2) == RANGE
        # positions up to 15 + 57 * 5 - 1 = 299 fit the rotary table, 58 steps do not
        assert h.begin_async([1], [15], [4], 58) == RANGE
        # all or nothing: 0 fits alone (7 more pages of 10 free), both do not
        assert h.begin_async([0, 1], [15, 15], [4, 4], 20) == OOM
        assert h.free() == f and h.seq(0)["pages"] == 1
        assert h.begin_async([0], [15], [4], 20) == OK
        assert h.seq(0)["pages"] == pages_for(15 + 20 * 5 + 1)
        assert h.verify([0], [15], [[1]]) == STATE
        assert h.verify([1], [15], [[1]], acc=[0], nxt=[3]) == OK  # sequence 1 is not in the loop
        h.end_async([0], [15], [16])  # a loop that ran no step
        assert h.seq(0)["pages"] == 1 and h.free() == f - 0 - (pages_for(17) - 1)
    finally:
        h.close()
