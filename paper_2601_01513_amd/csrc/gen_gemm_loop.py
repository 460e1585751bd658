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
  - LDS (160 KB) holds the A panels in two stages (32 KB each, at 0) and the
    B panels in three (at 64 KB): B is the weight matrix, streamed from HBM,
    so its loads are issued two panels ahead; A (activations, mostly cache
    hits) one panel ahead. Rows are 128 bytes, chunk c of row r at
    c ^ ((r/2) % 8). The stage of panel k is k % 2 for A and k % 3 for B, so
    the loop is unrolled over the 6-panel cycle (each body names its stages
    as immediate offsets: rdA / rdB with stage * 32 KB, rdC = rdB + 64 KB
    for the third B stage);
  - LDS-direct global loads (`global_load_lds_dwordx4`, 1 KB per instruction
    and wave; M0 holds the wave's LDS destination), 8 per operand, lane and
    panel.

Schedule of panel k (16 MFMAs per k-step, each about 32 cycles of the
SIMD's matrix core; other instructions are issued between them):
  - k-step 0: A(k + 1)'s 8 loads, k-step 1: B(k + 2)'s 8 loads, one after
    each MFMA (each M0 written one MFMA ahead); the fragments of the
    following k-step are read from MFMA 1 on;
  - k-step 2: the global offsets advance by one panel (128 bytes);
  - k-step 3: after 12 MFMAs, wait for this lane's loads of panel k + 1
    (vmcnt(8): A(k+1) and the older B(k+1) done, B(k+2) may still fly) and
    for its fragment reads, then barrier (every wave's loads of panel k + 1
    are in LDS, and no wave still reads the stages that panel k + 2's loads
    overwrite); the last 4 MFMAs cover the reads of panel k + 1's first
    k-step.
Before each MFMA, lgkmcnt(N) waits exactly for its two fragments (LDS reads
complete in issue order). The second-to-last panel loads only A, the last
panel nothing and has no barrier.
"""
from __future__ import annotations

import os
import re
import sys

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gemm_loop_4w.inc")

NSTEP = 4        # 16-wide k-steps per 64-wide panel
STG = 32768      # bytes of one stage of one operand (256 rows x 128 bytes)
B_BASE = 65536   # byte offset of the B stages
FRAG = 4096      # bytes between 32-row fragments
HANDOFF = 12   # MFMAs of the last k-step issued before the barrier
# Read order of a fragment set: the first MFMA needs A0 and B0, the next
# three B1..B3, then A1..A3 one per row of four MFMAs.
READ_ORDER = [('a', 0), ('b', 0), ('b', 1), ('b', 2), ('b', 3), ('a', 1), ('a', 2), ('a', 3)]
MFMA_ORDER = [(i, j) for i in range(4) for j in range(4)]


class Stream:
    def __init__(self):
        self.lines, self.lgkm = [], []

    def op(self, s):
        self.lines.append(s)

    def read(self, fset, kind, idx, step, ast, bst):
        if kind == 'a':
            self.op(f'ds_read_b128 %[fa{fset}{idx}], %[rdA{step}] offset:{ast * STG + idx * FRAG}')
        elif bst < 2:
            self.op(f'ds_read_b128 %[fb{fset}{idx}], %[rdB{step}] offset:{bst * STG + idx * FRAG}')
        else:
            self.op(f'ds_read_b128 %[fb{fset}{idx}], %[rdC{step}] offset:{idx * FRAG}')
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


def loads(kind, stage):
    base = 0 if kind == 'A' else B_BASE
    return [(f's_add_u32 m0, %[mw], {base + stage * STG + i * FRAG}',
             f'global_load_lds_dwordx4 %[d{kind}{i}], %[p{kind.lower()}]') for i in range(8)]


ADV_A = [f'v_add_u32 %[dA{i}], 128, %[dA{i}]' for i in range(8)]
ADV_B = [f'v_add_u32 %[dB{i}], 128, %[dB{i}]' for i in range(8)]


def publish(e, vm):
    """Panel hand-off: this lane's loads down to vm in flight, then barrier."""
    e.op(f's_waitcnt vmcnt({vm})')
    e.op('s_barrier')


def panel(e, p, kind):
    """Panel of phase p (A stage p % 2, B stage p % 3). kind: 'full' (loads
    A(k+1), B(k+2)), 'pre' (loads A(k+1) only), 'last' (no loads)."""
    a, b = p % 2, p % 3
    an, bn = (p + 1) % 2, (p + 1) % 3
    todo = []
    if kind in ('full', 'pre'):
        todo += loads('A', an)
    if kind == 'full':
        todo += loads('B', (p + 2) % 3)
    for s in range(NSTEP):
        fs, other = s & 1, (s & 1) ^ 1
        reads = [(other, k, idx, s + 1, a, b) for k, idx in READ_ORDER] if s + 1 < NSTEP else []
        handoff = s == NSTEP - 1 and kind != 'last'
        mine = todo[:8] if s < 2 else []
        todo = todo[8:] if s < 2 else todo
        m0_set = False
        for n, (i, j) in enumerate(MFMA_ORDER):
            if handoff and n == HANDOFF:
                e.drain()
                publish(e, 8 if kind == 'full' else 0)
            e.mfma(fs, i, j)
            if 1 <= n <= len(reads):
                e.read(*reads[n - 1])
            if s == 2 and kind == 'full':
                e.op((ADV_A + ADV_B)[n])
            if s == 2 and kind == 'pre' and n < 8:
                e.op(ADV_A[n])
            if handoff and n >= HANDOFF:
                per = -(-len(READ_ORDER) // (16 - HANDOFF))
                for k, idx in READ_ORDER[(n - HANDOFF) * per:(n - HANDOFF + 1) * per]:
                    e.read(0, k, idx, 0, an, bn)
            if mine and m0_set and n >= 1:
                e.op(mine.pop(0)[1])
                m0_set = False
            if mine and not m0_set:
                e.op(mine[0][0])
                m0_set = True
        assert not mine


def generate():
    e = Stream()
    for m0, ld in loads('A', 0) + loads('B', 0):
        e.op(m0); e.op('s_nop 0'); e.op(ld)
    e.op('s_cmp_eq_u32 %[n], 1')
    e.op('s_cbranch_scc1 L_one_%=')
    for a in ADV_B:
        e.op(a)
    for m0, ld in loads('B', 1):
        e.op(m0); e.op('s_nop 0'); e.op(ld)
    e.op('s_waitcnt vmcnt(8)')
    e.op('s_barrier')
    for x in ADV_A + ADV_B:
        e.op(x)
    for k, idx in READ_ORDER:
        e.read(0, k, idx, 0, 0, 0)
    entry = list(e.lgkm)
    e.op('s_cmp_eq_u32 %[n], 2')
    e.op('s_cbranch_scc1 L_pre0_%=')
    e.op('L_loop_%=:')
    for p in range(6):
        e.lgkm = list(entry)
        panel(e, p, 'full')
        e.op('s_sub_u32 %[n], %[n], 1')
        e.op('s_cmp_eq_u32 %[n], 2')
        e.op(f's_cbranch_scc1 L_pre{(p + 1) % 6}_%=')
    e.op('s_branch L_loop_%=')
    e.op('L_one_%=:')
    e.op('s_waitcnt vmcnt(0)')
    e.op('s_barrier')
    for k, idx in READ_ORDER:
        e.read(0, k, idx, 0, 0, 0)
    e.op('s_branch L_last0_%=')
    for p in range(6):
        e.op(f'L_pre{p}_%=:')
        e.lgkm = list(entry)
        panel(e, p, 'pre')
        e.op(f's_branch L_last{(p + 1) % 6}_%=')
    for p in range(6):
        e.op(f'L_last{p}_%=:')
        e.lgkm = list(entry)
        panel(e, p, 'last')
        e.op('s_branch L_end_%=')
    e.op('L_end_%=:')
    for _ in range(3):
        e.op('s_nop 7')
    return e.lines


def check(lines, nmax=14):
    """Interprets the stream for 1..nmax panels. Every MFMA must read
    fragments of its own (panel, k-step), with their reads complete; every
    fragment read must come from a stage whose loads completed (vmcnt) and
    were published by a barrier, and the 32 rows it reads must hold the panel
    its k-step belongs to (load slot q of the four waves fills rows
    32 q .. + 31: fragment i is slot i for waves in the first row (A) or
    column (B) half and slot 4 + i for the others; each slot's offset
    advances on its own); a load may not overwrite a stage that this wave
    has read since the last barrier, or whose reads were still in flight at
    it; each load's M0 must be the slot of its own row block; the MFMAs must
    walk panels 0..n-1, k-steps 0..3."""
    labels = {l[:-1]: i for i, l in enumerate(lines) if re.match(r'L_\w+_%=:$', l)}
    for n0 in range(1, nmax + 1):
        n, pc, scc = n0, 0, False
        koff = {(k, i): 0 for k in 'AB' for i in range(8)}
        stage, inflight = {}, []
        tag, pending, done, src = {}, [], set(), {}
        seen, busy, m0 = [], set(), None
        steps = 0
        while pc < len(lines):
            steps += 1
            assert steps < 400000
            l = lines[pc]; pc += 1
            if l.endswith(':') or l.startswith('s_nop'):
                continue
            m = re.match(r's_add_u32 m0, %\[mw\], (\d+)$', l)
            if m:
                off = int(m.group(1))
                kind = 'B' if off >= B_BASE else 'A'
                rel = off - (B_BASE if kind == 'B' else 0)
                m0 = (kind, rel // STG, (rel % STG) // FRAG)
                assert (kind == 'A' and m0[1] < 2) or (kind == 'B' and m0[1] < 3)
                continue
            m = re.match(r'global_load_lds_dwordx4 %\[d([AB])(\d)\], %\[p([ab])\]$', l)
            if m:
                kind = m.group(1)
                assert m0 and m0[0] == kind and m0[2] == int(m.group(2)) and m.group(3) == kind.lower(), (l, m0)
                st, slot = m0[1], m0[2]
                assert (kind, st) not in busy, ('load over a stage in use', l)
                inflight.append((kind, st, slot, koff[(kind, slot)]))
                stage[(kind, st, slot)] = (koff[(kind, slot)], 'pending')
                m0 = None
                continue
            m = re.match(r'v_add_u32 %\[d([AB])(\d)\], 128, %\[d\1\2\]$', l)
            if m:
                koff[(m.group(1), int(m.group(2)))] += 1
                continue
            m = re.match(r's_waitcnt vmcnt\((\d+)\)$', l)
            if m:
                keep = int(m.group(1))
                while len(inflight) > keep:
                    kind, st, slot, p = inflight.pop(0)
                    if stage[(kind, st, slot)] == (p, 'pending'):
                        stage[(kind, st, slot)] = (p, 'landed')
                continue
            if l == 's_barrier':
                for k, v in list(stage.items()):
                    if v[1] == 'landed':
                        stage[k] = (v[0], 'visible')
                busy = {src[r] for r in pending}
                continue
            m = re.match(r'ds_read_b128 %\[(f([ab])\d(\d))\], %\[rd([ABC])(\d)\] offset:(\d+)$', l)
            if m:
                reg, idx, base, step, off = m.group(1), int(m.group(3)), m.group(4), int(m.group(5)), int(m.group(6))
                kind = 'A' if base == 'A' else 'B'
                assert m.group(2) == kind.lower()
                st = 2 if base == 'C' else off // STG
                assert off % STG == idx * FRAG
                p, state = stage[(kind, st, idx)]
                p2, state2 = stage[(kind, st, 4 + idx)]
                assert state == state2 == 'visible', ('read of an unpublished stage', l, state, state2)
                assert p == p2
                tag[reg] = (p, step); src[reg] = (kind, st)
                pending.append(reg); done.discard(reg)
                busy.add((kind, st))
                continue
            m = re.match(r's_waitcnt lgkmcnt\((\d+)\)$', l)
            if m:
                while len(pending) > int(m.group(1)):
                    done.add(pending.pop(0))
                continue
            m = re.match(r'v_mfma_f32_32x32x16_f16 %\[c(\d)(\d)\], %\[(fa\d(\d))\], %\[(fb\d(\d))\], %\[c\1\2\]$', l)
            if m:
                a_, b_ = m.group(3), m.group(5)
                assert m.group(4) == m.group(1) and m.group(6) == m.group(2)
                assert a_ in done and b_ in done, ('fragment read not complete', l)
                assert tag[a_] == tag[b_], (tag[a_], tag[b_], l)
                seen.append(tag[a_])
                continue
            m = re.match(r's_cmp_eq_u32 %\[n\], (\d)$', l)
            if m:
                scc = n == int(m.group(1)); continue
            if l == 's_sub_u32 %[n], %[n], 1':
                n -= 1; continue
            m = re.match(r's_cbranch_scc1 (L_\w+_%=)$', l)
            if m:
                pc = labels[m.group(1)] if scc else pc; continue
            m = re.match(r's_branch (L_\w+_%=)$', l)
            if m:
                pc = labels[m.group(1)]; continue
            raise AssertionError(f'unknown: {l}')
        want = [(p, s) for p in range(n0) for s in range(NSTEP) for _ in range(16)]
        assert seen == want, (n0, seen[:5], len(seen))
        assert not inflight
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
