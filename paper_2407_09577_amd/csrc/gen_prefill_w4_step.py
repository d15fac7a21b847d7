"""Writes prefill_w4_step.inc, the k-block step of the 4-wave 256 x 256 prefill tile.

The tile (2 x 2 waves of 128 x 128, one wave per SIMD) walks K in 32-deep blocks.  One
block of one wave is 64 matrix-core ops (8 x 8 fragments of 16 x 16 x 32) plus, for the
RMS kinds, 4 Gram ops that take the squares of the wave's share of row blocks.  Between
them the step issues the next block's 16 fragment reads from LDS, the 8 LDS-DMA transfers
of the block STAGES ahead, and the address arithmetic for the next step.  The compiler does
not keep such a schedule (nor the accumulators in AGPRs with one wave per SIMD), so the
step is one inline-asm sequence whose operands the compiler still allocates: this script
writes it, with the C++ wrappers that bind the operands.

Schedule (op m = 0..63 of the block, i-major: op m multiplies column fragment m / 8 with
row fragment m % 8): read r after op 4 r; transfer n's M0 arithmetic after op 8 n + 2, the
M0 move and the transfer after op 8 n + 3, its offset increment after op 8 n + 6.  Chosen
by measurement on MI355X among spreads of the same instructions (Llama-7B QKV shape).

Hazards the sequence covers itself: it starts with 5 wait states (earlier VALU and
accumulator writes); fragment reads land before it ends (lgkmcnt(0)), so the compiler may
move the outputs freely; M0 is written only by an s_mov immediately before its transfer;
the SCC writes of the address arithmetic are declared.  The caller inserts the wait states
between the last step and the first read of the accumulators.

Regenerate after editing:  python paper_2407_09577_amd/csrc/gen_prefill_w4_step.py
"""
import os

FM = FN = 8          # 16-row / 16-column fragments per wave (128 x 128 wave tile)
TW = 4               # row blocks whose statistics a wave takes (FM / WN, WN = 2)
NL = 8               # LDS-DMA transfers per wave per k block (32 fragments / 4 waves)
NA = 4               # of them activation fragments (16 row blocks / 4 waves)
STAGE = 0x8000       # bytes of one ring slot (32 fragments of 1 KiB)
SLOTS_MASK = 0x18000  # four slots
READ_EVERY = 4
LOAD_EVERY, LOAD_M0, LOAD_ISSUE, LOAD_ADVANCE = 8, 2, 3, 6


class Ops:
    """Operand numbering of one variant: outputs first, then inputs, as inline asm counts them."""

    def __init__(self, gram, full):
        self.outs, self.ins, self.idx = [], [], {}
        for t in range(FN * FM):
            self._out(f"acc{t}", f'"+a"(acc[{t // FM}][{t % FM}])')
        if gram:
            for t in range(TW):
                self._out(f"g{t}", f'"+v"(g[{t}])')
        if full:
            for r in range(8):
                self._out(f"na{r}", f'"=&v"(na[{r}])')
            for q in range(8):
                self._out(f"nw{q}", f'"=&v"(nw[{q}])')
            for i in range(NL):
                self._out(f"vo{i}", f'"+v"(vo[{i}])')
            self._out("sn", '"+s"(slot_n)')
            self._out("sl", '"+s"(slot_l)')
            self._out("va", '"=&v"(va_t)')
            self._out("vw", '"=&v"(vw_t)')
            self._out("m0t", '"=&s"(m0_t)')
        ins = [(f"ca{r}", f'"v"(ca[{r}])') for r in range(8)] + [(f"cw{q}", f'"v"(cw[{q}])') for q in range(8)]
        if full:
            ins += [("aconst", '"v"(aconst)'), ("wconst", '"v"(wconst)'), ("mbase", '"s"(mbase)'),
                    ("dw", '"s"(dw)'), ("rsa", '"s"(rsa)'), ("rsw", '"s"(rsw)')]
        for j, (k, c) in enumerate(ins):
            self.idx[k] = len(self.outs) + j
            self.ins.append(c)

    def _out(self, k, c):
        self.idx[k] = len(self.outs)
        self.outs.append(c)

    def __getitem__(self, k):
        return f"%{self.idx[k]}"


def body(o, wnc, gram, full):
    lines = ["s_nop 4"]
    if full:
        lines += [f"v_add_u32 {o['va']}, {o['sn']}, {o['aconst']}", f"v_add_u32 {o['vw']}, {o['sn']}, {o['wconst']}"]
    if gram:
        for t in range(TW):
            j = wnc + 2 * t  # row blocks wnc, wnc + 2, ... of the wave's eight
            lines.append(f"v_mfma_f32_16x16x32_bf16 {o[f'g{t}']}, {o[f'ca{j}']}, {o[f'ca{j}']}, {o[f'g{t}']}")
    after = {}
    if full:
        for r in range(16):
            dst, addr, off = (o[f"na{r}"], o["va"], r) if r < 8 else (o[f"nw{r - 8}"], o["vw"], r - 8)
            after.setdefault(READ_EVERY * r, []).append(f"ds_read_b128 {dst}, {addr} offset:{off * 1024}")
        for n in range(NL):
            base = LOAD_EVERY * n
            after.setdefault(base + LOAD_M0, []).extend(
                [f"s_add_u32 {o['m0t']}, {o['sl']}, {o['mbase']}", f"s_add_u32 {o['m0t']}, {o['m0t']}, {n * 4096}"])
            after.setdefault(base + LOAD_ISSUE, []).extend(
                [f"s_mov_b32 m0, {o['m0t']}",
                 f"buffer_load_dwordx4 {o[f'vo{n}']}, {o['rsa'] if n < NA else o['rsw']}, 0 offen lds"])
            step = "64" if n < NA else o["dw"]  # 32 bf16 of an activation row; one k block of W*
            after.setdefault(base + LOAD_ADVANCE, []).append(f"v_add_u32 {o[f'vo{n}']}, {step}, {o[f'vo{n}']}")
        assert max(after) < FN * FM
    for m in range(FN * FM):
        i, j = m // FM, m % FM
        lines.append(f"v_mfma_f32_16x16x32_bf16 {o[f'acc{m}']}, {o[f'cw{i}']}, {o[f'ca{j}']}, {o[f'acc{m}']}")
        lines += after.get(m, [])
    if full:
        lines += [f"s_add_u32 {o['sn']}, {o['sn']}, {STAGE:#x}", f"s_and_b32 {o['sn']}, {o['sn']}, {SLOTS_MASK:#x}",
                  f"s_add_u32 {o['sl']}, {o['sl']}, {STAGE:#x}", f"s_and_b32 {o['sl']}, {o['sl']}, {SLOTS_MASK:#x}",
                  "s_waitcnt lgkmcnt(0)"]
    return "\\n\\t".join(lines)


def generate():
    out = ["// Generated by gen_prefill_w4_step.py (see there); do not edit.", "", "namespace fn {", ""]
    for gram in (True, False):
        for full in (True, False):
            for wnc in ((0, 1) if gram else (0,)):
                o = Ops(gram, full)
                name = f"w4_step_{'full' if full else 'last'}_{'gram' if gram else 'plain'}{wnc if gram else ''}"
                if full:
                    sig = ("f32x4 (&acc)[8][8], f32x4 (&g)[4], u32x4 (&na)[8], u32x4 (&nw)[8], const u32x4 (&ca)[8],\n"
                           "    const u32x4 (&cw)[8], unsigned (&vo)[8], unsigned& slot_n, unsigned& slot_l, unsigned aconst,\n"
                           "    unsigned wconst, unsigned mbase, unsigned dw, i32x4 rsa, i32x4 rsw")
                    pre, clob = "  unsigned va_t, vw_t, m0_t;\n", '"scc", "memory"'
                else:
                    sig = "f32x4 (&acc)[8][8], f32x4 (&g)[4], const u32x4 (&ca)[8], const u32x4 (&cw)[8]"
                    pre, clob = "", '"memory"'
                out.append(f"__device__ __forceinline__ void {name}(\n    {sig}) {{\n{pre}"
                           f"  asm volatile(\"{body(o, wnc, gram, full)}\"\n"
                           f"      : {', '.join(o.outs)}\n      : {', '.join(o.ins)}\n      : {clob});\n}}\n")
    out.append("}  // namespace fn")
    return "\n".join(out) + "\n"


if __name__ == "__main__":
    open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "prefill_w4_step.inc"), "w").write(generate())
