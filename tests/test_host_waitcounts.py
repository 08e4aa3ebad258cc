"""The hand-counted vmcnt waits of the direct-to-LDS pipelines hold in the
code the compiler emits (host-only: compiles the kernels to gfx950 assembly).

Three designs wait for loads that land in LDS by counting, rather than by a
full vmcnt(0): the score GEMM (a stage of training rows has landed once no
more than 28 / 18 later loads are outstanding), the direct-load projection
(a stage has landed once no more than one stage's loads are outstanding) and
the weight-gradient tile (once no more than two later stages' loads are).
Direct loads are invisible to the compiler's own wait insertion, so these
counts are only right while the compiled load order is the designed one.
These tests read that order from the assembly of this build.
"""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2609_38767_amd import build as B

HAND_BARRIER = re.compile(r"s_waitcnt lgkmcnt\(0\)")


def _asm(src):
    out = os.path.join(tempfile.mkdtemp(prefix="dattri_asm_"), src + ".s")
    cmd = [B.HIPCC] + B.COMMON + B.DEVICE + ["-x", "hip", "--offload-device-only", "-S",
                                            os.path.join(B.CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read().splitlines()


def _body(lines, symbol_prefix):
    start = next(i for i, l in enumerate(lines) if l.startswith(symbol_prefix) and ":" in l)
    body = []
    for l in lines[start + 1:]:
        body.append(l.strip())
        if l.strip() == "s_endpgm":
            break
    return body


def _events(body):
    """Vector memory ops in text order: 'D' direct load into LDS, 'R' load
    into registers, 'S' store; and ('W', n) for a hand-counted wait (a vmcnt
    wait followed by the inline LDS-drain-and-barrier sequence)."""
    ev = []
    for i, t in enumerate(body):
        if t.startswith(("buffer_load", "global_load")):
            ev.append("D" if t.endswith(" lds") else "R")
        elif t.startswith(("buffer_store", "global_store")):
            ev.append("S")
        else:
            m = re.match(r"s_waitcnt vmcnt\((\d+)\)$", t)
            if m and any(HAND_BARRIER.search(x) for x in body[i + 1:i + 4]) and \
                    any(x == "s_barrier" for x in body[i + 1:i + 5]):
                ev.append(("W", int(m.group(1))))
    return ev


@pytest.fixture(scope="module")
def score_asm():
    return _asm("score_big.hip")


def test_score_gemm_stage_waits(score_asm):
    # Design: the prologue loads stages 0 and 1 of training rows (8 direct
    # loads each) and 5 K steps of query fragments (20 register loads), then
    # waits with vmcnt(28) for stage 0.  Stage kk loads stage kk + 2 (8 direct
    # loads, 6 before and 2 after its wait) and waits with vmcnt(18) for stage
    # kk + 1.  At every wait, the loads issued after the awaited stage's last
    # direct load must number at least the wait's count.  The text of the
    # kernel is itself an execution path (prologue, one pass of the three-stage
    # loop, both remainder stages); the last stage's wait guards a stage past
    # the end that is never read.
    ev = _events(_body(score_asm, "_ZN6dattri21score_gemm_256_kernel"))
    waits = [i for i, e in enumerate(ev) if isinstance(e, tuple)]
    assert [ev[i][1] for i in waits] == [28, 18, 18, 18, 18, 18], [ev[i] for i in waits]
    d_pos = [i for i, e in enumerate(ev) if e == "D"]
    ops = lambda a, b: sum(1 for e in ev[a + 1:b] if e in ("D", "R", "S"))
    checked = 0
    for w, i in enumerate(waits[:-1]):  # the final stage's wait guards nothing read
        group = w  # the prologue wait awaits stage 0, stage kk's wait stage kk + 1
        last_d = d_pos[8 * group + 7]
        assert last_d < i, (w, last_d, i)
        assert ops(last_d, i) >= ev[i][1], (w, ops(last_d, i), ev[i][1])
        checked += 1
    assert checked == 5


@pytest.fixture(scope="module")
def factored_asm():
    return _asm("factored.hip")


@pytest.mark.parametrize("na,nb", [(2, 2), (4, 2), (6, 2), (2, 4), (4, 4)])
def test_direct_load_projection_waits(factored_asm, na, nb):
    # Design (project_rows_dma, once for the input side with NA map tiles and
    # once for the output side with NB, inlined; the member loop is not
    # unrolled): every stage issues exactly k = 8 row-group loads + NT / 2
    # map-fragment loads, all direct loads, two stages before the stage loop
    # and one per iteration after the stage's compute; the wait at the top of
    # iteration s is vmcnt(k) (vmcnt(0) on the last).  So the text holds
    # exactly 3 k_A + 3 k_B direct loads, no other load or store among them,
    # and the kernel's vmcnt waits are k_A, k_B and 0 only.
    sym = f"_ZN6dattri15factored_kernelILi2ELb1ELi4ELi{na}ELi{nb}E"
    body = _body(factored_asm, sym)
    ev = [e for e in _events(body) if isinstance(e, str)]
    k_a, k_b = 8 + na // 2, 8 + nb // 2
    d_pos = [i for i, e in enumerate(ev) if e == "D"]
    assert len(d_pos) == 3 * (k_a + k_b), (len(d_pos), k_a, k_b)
    assert all(e == "D" for e in ev[d_pos[0]:d_pos[-1] + 1]), "".join(ev)
    counts = {int(m.group(1)) for t in body for m in [re.match(r"s_waitcnt vmcnt\((\d+)\)$", t)] if m}
    assert counts == {0, k_a, k_b}, (counts, k_a, k_b)


@pytest.fixture(scope="module")
def kfac_asm():
    return _asm("kfac.hip")


@pytest.mark.parametrize("nt,rt", [(2, 4), (4, 2)])
def test_direct_load_factor_sum_waits(kfac_asm, nt, rt):
    # The factor-sum pass's bf16 instances stream rows by the same
    # project_rows_dma (inlined once per kernel, RT row tiles per wave): each
    # stage issues k = 2 RT row-group loads + NT / 2 map-fragment loads, the
    # text holds 3 k direct loads with nothing else among them, and the only
    # vmcnt waits are k and 0.
    body = _body(kfac_asm, f"_ZN6dattri11fsum_kernelILi2ELb1ELi{nt}E")
    ev = [e for e in _events(body) if isinstance(e, str)]
    k = 2 * rt + nt // 2
    d_pos = [i for i, e in enumerate(ev) if e == "D"]
    assert len(d_pos) == 3 * k, (len(d_pos), k)
    assert all(e == "D" for e in ev[d_pos[0]:d_pos[-1] + 1]), "".join(ev)
    counts = {int(m.group(1)) for t in body for m in [re.match(r"s_waitcnt vmcnt\((\d+)\)$", t)] if m}
    assert counts <= {0, k} and k in counts, (counts, k)


@pytest.mark.parametrize("src,sym", [("gradient_tr.hip", "_ZN6dattri18gradient_tr_kernel"),
                                     ("xone.hip", "_ZN6dattri11xone_kernel"),
                                     ("gfused.hip", "_ZN6dattri13gfused_kernelILi1E"),
                                     ("gfused.hip", "_ZN6dattri13gfused_kernelILi2E"),
                                     ("gfused.hip", "_ZN6dattri13gfused_kernelILi4E"),
                                     ("crossgram.hip", "_ZN6dattri12ghost_kernelILi2E")])
def test_direct_load_gradient_tile_waits(src, sym):
    # Design (g_tile_dma, inlined once per tile the kernel forms; the
    # factorized cross-Gram tile ghost_tile_dma has the same ring): every
    # stage is 4 direct loads per wave (2 per side), up to three stages issued
    # before the stage loop and one per iteration after the stage barrier; the
    # hand wait before stage k's barrier is vmcnt(4 x min(2, stages after k))
    # = 8, 4 or 0.  The transposing LDS reads are inline assembly, so the
    # compiler inserts no vmcnt wait of its own between a barrier and the
    # reads that follow it (a wait there would drain the ring each stage).
    body = _body(_asm(src), sym)
    ev = _events(body)
    hand = {e[1] for e in ev if isinstance(e, tuple)}
    assert 8 in hand and hand <= {0, 4, 8}, hand
    n_d = sum(1 for e in ev if e == "D")
    assert n_d > 0 and n_d % 4 == 0, n_d
    if src == "crossgram.hip":  # its register-staged form shares the kernel; reads not checked
        return
    reads = [i for i, t in enumerate(body) if t.startswith("ds_read_b64_tr_b16")]
    assert reads
    for i in reads:
        j = i - 1
        while j >= 0 and body[j] != "s_barrier" and not body[j].startswith("ds_read_b64_tr_b16"):
            assert not body[j].startswith("s_waitcnt vmcnt"), (i, body[j])
            j -= 1
