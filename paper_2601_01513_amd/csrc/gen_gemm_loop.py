"""Writes gemm_loop_4w.inc: the explicitly ordered K loop of the four-wave
256 x 256 MFMA GEMM tile (kernels_gemm.hip, mainloop_4w), and checks it.

The loop is one inline-assembly block, so the compiler neither reorders it
nor inserts waits into it: every wait below is placed here, and `check`
replays the stream to prove the placement. Run from the repository root:

    python paper_2601_01513_amd/csrc/gen_gemm_loop.py          # rewrite + check
    python paper_2601_01513_amd/csrc/gen_gemm_loop.py --check  # check only

Shape of the work (per wave, one of four; wave w owns output rows
128 (w / 2) .. + 127 and columns 128 (w % 2) .. + 127 of the tile):
  - accumulators c{i}{j}: 4 x 4 blocks of 32 x 32 (v_mfma_f32_32x32x16_f16,
    256 accumulation registers);
  - a K panel is 64 wide = four 16-wide k-steps; k-step s uses fragments
    fa{set}{i} (rows of A) and fb{set}{j} (rows of B), 16 bytes per lane,
    read from LDS; two fragment sets alternate between k-steps;
  - LDS holds two panels (stages): A rows at stage * 32 KB, B rows at
    64 KB + stage * 32 KB, 128-byte rows, chunk c of row r at c ^ ((r/2) % 8);
  - the next panel streams into the other stage with LDS-direct global loads
    (`global_load_lds_dwordx4`, 1 KB per instruction and wave; M0 holds the
    wave's LDS destination), 8 for A and 8 for B per lane and panel.

Schedule of one panel (16 MFMAs per k-step, each about 32 cycles of the
SIMD's matrix core; other instructions are issued between them):
  - k-steps 0 and 1: the next panel's 16 loads, one after each MFMA; the
    fragments of the following k-step are read from MFMA 1 on;
  - k-step 2: the global offsets advance by one panel (128 bytes);
  - k-step 3: after 12 MFMAs, wait for this lane's loads (vmcnt(0)) and for
    its fragment reads, then barrier (every wave's loads of the next panel
    are in LDS, and no wave still reads the current stage, which the next
    panel's loads will overwrite); the last 4 MFMAs cover the reads of the
    next panel's first k-step.
Before each MFMA, lgkmcnt(N) waits exactly for its two fragments (LDS reads
complete in issue order). A last panel issues no loads and has no barrier.
"""
from __future__ import annotations

import os
import re
import sys

NSTEP = 4            # 16-wide k-steps per 64-wide panel
A_STAGE = 32768      # bytes of one stage's A (or B) rows
B_BASE = 65536       # byte offset of the B rows
FRAG = 4096          # bytes between 32-row fragments
HANDOFF = 12         # MFMAs of the last k-step issued before the barrier
LOADS_PER_PANEL = 16
# Read order of a fragment set: the first MFMA needs A0 and B0, the next
# three B1..B3, then A1..A3 one per row of four MFMAs.
READ_ORDER = [('a', 0), ('b', 0), ('b', 1), ('b', 2), ('b', 3), ('a', 1), ('a', 2), ('a', 3)]
MFMA_ORDER = [(i, j) for i in range(4) for j in range(4)]

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gemm_loop_4w.inc")


class Stream:
    def __init__(self):
        self.lines = []
        self.lgkm = []  # outstanding fragment reads, issue order

    def op(self, s):
        self.lines.append(s)

    def read(self, fset, kind, idx, step, stage):
        self.op(f'ds_read_b128 %[f{kind}{fset}{idx}], %[rd{kind.upper()}{step}] '
                f'offset:{idx * FRAG + stage * A_STAGE}')
        self.lgkm.append((fset, kind, idx))

    def need(self, fset, kind, idx):
        if (fset, kind, idx) in self.lgkm:
            pos = self.lgkm.index((fset, kind, idx))
            self.op(f's_waitcnt lgkmcnt({len(self.lgkm) - pos - 1})')
            self.lgkm = self.lgkm[pos + 1:]

    def drain(self):
        if self.lgkm:
            self.op('s_waitcnt lgkmcnt(0)')
            self.lgkm = []

    def mfma(self, fset, i, j):
        self.need(fset, 'a', i)
        self.need(fset, 'b', j)
        self.op(f'v_mfma_f32_32x32x16_f16 %[c{i}{j}], %[fa{fset}{i}], %[fb{fset}{j}], %[c{i}{j}]')


def loads(stage):
    """(M0 write, load) pairs that fill LDS stage `stage` with a panel."""
    out = []
    for kind, base in (('A', 0), ('B', B_BASE)):
        for i in range(8):
            out.append((f's_add_u32 m0, %[mw], {base + stage * A_STAGE + i * FRAG}',
                        f'global_load_lds_dwordx4 %[d{kind}{i}], %[p{kind.lower()}]'))
    return out


ADVANCE = [f'v_add_u32 %[d{k}{i}], 128, %[d{k}{i}]' for k in 'AB' for i in range(8)]


def panel(e, cur, last):
    """One panel from stage `cur`; fragment set 0 holds (or is reading) k-step 0."""
    nxt = 1 - cur
    todo = [] if last else loads(nxt)
    for s in range(NSTEP):
        fs, other = s & 1, (s & 1) ^ 1
        reads = [(other, k, idx, s + 1, cur) for k, idx in READ_ORDER] if s + 1 < NSTEP else []
        handoff = s == NSTEP - 1 and not last
        mine = todo[:8] if s < 2 else []
        todo = todo[8:] if s < 2 else todo
        m0_set = False
        for n, (i, j) in enumerate(MFMA_ORDER):
            if handoff and n == HANDOFF:
                e.drain()
                e.op('s_waitcnt vmcnt(0)')
                e.op('s_barrier')
            e.mfma(fs, i, j)
            if 1 <= n <= len(reads):
                e.read(*reads[n - 1])
            if s == 2 and not last:
                e.op(ADVANCE[n])
            if handoff and n >= HANDOFF:
                per = -(-len(READ_ORDER) // (16 - HANDOFF))
                for k, idx in READ_ORDER[(n - HANDOFF) * per:(n - HANDOFF + 1) * per]:
                    e.read(0, k, idx, 0, nxt)
            # each load one MFMA after the write of its M0
            if mine and m0_set and n >= 1:
                e.op(mine.pop(0)[1])
                m0_set = False
            if mine and not m0_set:
                e.op(mine[0][0])
                m0_set = True
        assert not mine


def generate():
    e = Stream()
    for m0, ld in loads(0):
        e.op(m0)
        e.op('s_nop 0')
        e.op(ld)
    e.op('s_waitcnt vmcnt(0)')
    e.op('s_barrier')
    for a in ADVANCE:
        e.op(a)
    for k, idx in READ_ORDER:
        e.read(0, k, idx, 0, 0)
    entry = list(e.lgkm)
    e.op('s_cmp_eq_u32 %[n], 1')
    e.op('s_cbranch_scc1 L_last0_%=')
    e.op('L_loop_%=:')
    panel(e, 0, False)
    e.op('s_sub_u32 %[n], %[n], 1')
    e.op('s_cmp_eq_u32 %[n], 1')
    e.op('s_cbranch_scc1 L_last1_%=')
    panel(e, 1, False)
    e.op('s_sub_u32 %[n], %[n], 1')
    e.op('s_cmp_eq_u32 %[n], 1')
    e.op('s_cbranch_scc1 L_last0_%=')
    e.op('s_branch L_loop_%=')
    e.op('L_last0_%=:')
    e.lgkm = list(entry)
    panel(e, 0, True)
    e.op('s_branch L_end_%=')
    e.op('L_last1_%=:')
    e.lgkm = list(entry)
    panel(e, 1, True)
    e.op('L_end_%=:')
    # the accumulators are read right after the block: let the last MFMAs
    # retire first
    for _ in range(3):
        e.op('s_nop 7')
    return e.lines


def check(lines, nmax=7):
    """Interprets the stream for 1..nmax panels. Every MFMA must read
    fragments of its own (panel, k-step), with their reads complete; every
    fragment read must come from a stage whose loads completed (vmcnt(0)) and
    were published by a barrier; a load may not overwrite a stage that this
    wave has read since the last barrier; each load's M0 must be the slot of
    its own row block, and the 32 rows a fragment reads must hold the panel
    its k-step belongs to (each load slot advances on its own); the MFMAs must walk panels 0..n-1, k-steps 0..3."""
    labels = {l[:-1]: i for i, l in enumerate(lines) if re.match(r'L_\w+_%=:$', l)}
    for n0 in range(1, nmax + 1):
        n, pc, scc = n0, 0, False
        koff = {(k, i): 0 for k in 'AB' for i in range(8)}
        stage, inflight = {}, []
        tag, pending, done, src = {}, [], set(), {}
        seen, read_since_bar, m0 = [], set(), None
        steps = 0
        while pc < len(lines):
            steps += 1
            assert steps < 100000, 'no exit'
            l = lines[pc]
            pc += 1
            if l.endswith(':') or l.startswith('s_nop'):
                continue
            m = re.match(r's_add_u32 m0, %\[mw\], (\d+)$', l)
            if m:
                off = int(m.group(1))
                assert off % FRAG == 0
                m0 = ('B' if off >= B_BASE else 'A', (off % B_BASE) // A_STAGE, (off % A_STAGE) // FRAG)
                continue
            m = re.match(r'global_load_lds_dwordx4 %\[d([AB])(\d)\], %\[p([ab])\]$', l)
            if m:
                kind = m.group(1)
                assert m0 is not None and m0[0] == kind and m0[2] == int(m.group(2)), (l, m0)
                assert m.group(3) == kind.lower(), l
                st, slot = m0[1], m0[2]
                assert (kind, st) not in read_since_bar, ('load over a stage still being read', l)
                inflight.append((kind, st, slot, koff[(kind, slot)]))
                stage[(kind, st, slot)] = (koff[(kind, slot)], 'pending')
                m0 = None
                continue
            m = re.match(r'v_add_u32 %\[d([AB])(\d)\], 128, %\[d\1\2\]$', l)
            if m:
                koff[(m.group(1), int(m.group(2)))] += 1
                continue
            if l == 's_waitcnt vmcnt(0)':
                for kind, st, slot, p in inflight:
                    stage[(kind, st, slot)] = (p, 'landed')
                inflight = []
                continue
            if l == 's_barrier':
                for k, v in list(stage.items()):
                    if v[1] == 'landed':
                        stage[k] = (v[0], 'visible')
                # a read still in flight at the barrier keeps its stage busy
                read_since_bar = {src[r] for r in pending}
                continue
            m = re.match(r'ds_read_b128 %\[(f([ab])\d(\d))\], %\[rd([AB])(\d)\] offset:(\d+)$', l)
            if m:
                reg, kind, idx = m.group(1), m.group(4), int(m.group(3))
                assert m.group(2) == kind.lower()
                step, off = int(m.group(5)), int(m.group(6))
                st = off // A_STAGE
                assert off % A_STAGE == idx * FRAG, l
                # load slot q of the four waves fills tile rows 32 q .. + 31:
                # fragment idx is slot idx for waves in the first row (A) or
                # column (B) half and slot 4 + idx for the others
                p, state = stage[(kind, st, idx)]
                p2, state2 = stage[(kind, st, 4 + idx)]
                assert state == state2 == 'visible', ('read of an unpublished stage', l, state, state2)
                assert p == p2, ('halves of a stage hold different panels', l)
                tag[reg] = (p, step)
                src[reg] = (kind, st)
                pending.append(reg)
                done.discard(reg)
                read_since_bar.add((kind, st))
                continue
            m = re.match(r's_waitcnt lgkmcnt\((\d+)\)$', l)
            if m:
                while len(pending) > int(m.group(1)):
                    done.add(pending.pop(0))
                continue
            m = re.match(r'v_mfma_f32_32x32x16_f16 %\[c(\d)(\d)\], %\[(fa\d(\d))\], %\[(fb\d(\d))\], %\[c\1\2\]$', l)
            if m:
                a, b = m.group(3), m.group(5)
                assert m.group(4) == m.group(1) and m.group(6) == m.group(2), l
                assert a in done and b in done, ('fragment read not complete', l)
                assert tag[a] == tag[b], (tag[a], tag[b], l)
                seen.append(tag[a])
                continue
            if l == 's_cmp_eq_u32 %[n], 1':
                scc = n == 1
                continue
            if l == 's_sub_u32 %[n], %[n], 1':
                n -= 1
                continue
            m = re.match(r's_cbranch_scc1 (L_\w+_%=)$', l)
            if m:
                pc = labels[m.group(1)] if scc else pc
                continue
            m = re.match(r's_branch (L_\w+_%=)$', l)
            if m:
                pc = labels[m.group(1)]
                continue
            raise AssertionError(f'unknown instruction: {l}')
        want = [(p, s) for p in range(n0) for s in range(NSTEP) for _ in range(16)]
        assert seen == want, (n0, 'panel / k-step order')
        assert not inflight, 'loads left in flight'
    return True


def render(lines):
    return ''.join('"' + l + '\\n"\n' for l in lines)


def main(argv):
    lines = generate()
    check(lines)
    text = ("// Generated by gen_gemm_loop.py (K loop of mainloop_4w); do not edit.\n"
            + render(lines))
    if '--check' in argv:
        with open(OUT) as f:
            if f.read() != text:
                raise SystemExit(f'{OUT} differs from the generator output')
        print('ok')
        return
    with open(OUT, 'w') as f:
        f.write(text)
    print(f'wrote {OUT}: {len(lines)} lines, {sum(1 for l in lines if "mfma" in l)} MFMAs')


if __name__ == '__main__':
    main(sys.argv[1:])
