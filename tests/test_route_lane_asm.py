"""The generated inner step of the lane-per-token router (route_lane_asm.h):
it is what its generator writes, and its instruction order keeps the DPP
read-after-write distance, checked on the text without a GPU."""
import importlib.util
import os
import re

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2410_12247_amd", "csrc")


def _gen():
    spec = importlib.util.spec_from_file_location("gen_route_lane",
                                                  os.path.join(CSRC, "gen_route_lane.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _blocks(text):
    """Instruction lists of the asm statements, one per expert count."""
    out = {}
    for m in re.finditer(r"void lane_stage_g(\d)\(.*?asm volatile\((.*?)\n        :", text, re.S):
        out[int(m.group(1))] = [l.strip().strip('"').replace("\\n\\t", "").strip()
                                for l in m.group(2).strip().split("\n")]
    return out


def test_header_matches_generator():
    with open(os.path.join(CSRC, "route_lane_asm.h")) as f:
        assert f.read() == _gen().render()


@pytest.mark.parametrize("G", [2, 4])
def test_dpp_operands_two_wait_states_after_valu_writes(G):
    """Every VGPR a DPP fma reads was last written by a VALU instruction at
    least two wait states earlier (each instruction counts one, s_nop N
    counts N + 1); values from before the block are at least that far."""
    ins = _blocks(_gen().render())[G]
    last_write = {}  # operand name -> wait-state clock of its VALU write
    clock = 0
    n_dpp = 0
    for line in ins:
        op = line.split()[0]
        if op == "s_nop":
            clock += int(line.split()[1]) + 1
            continue
        args = re.findall(r"%\[(\w+)\]", line)
        if op == "v_fmac_f32_dpp":
            n_dpp += 1
            for a in args:  # acc (read and written), router register, temporary
                written = last_write.get(a, -10)
                assert clock - written - 1 >= 2, (G, line, clock, written)
            last_write[args[0]] = clock
        elif op in ("v_lshlrev_b32", "v_and_b32"):
            last_write[args[0]] = clock
        else:
            assert op in ("ds_read_b128", "s_waitcnt"), line
        clock += 1
    assert n_dpp == 64 * G
    # the first DPP instruction is at least two wait states into the block
    first = next(i for i, l in enumerate(ins) if l.startswith("v_fmac_f32_dpp"))
    pre = sum(int(l.split()[1]) + 1 if l.startswith("s_nop") else 1 for l in ins[:first])
    assert pre >= 2


@pytest.mark.parametrize("G", [2, 4])
def test_fma_order_follows_h(G):
    """Each accumulator takes h = 4 j + c in ascending order: router register
    c with row_newbcast:j, times the widened x_h (low half of dword h / 2 for
    even h, high half for odd h)."""
    ins = _blocks(_gen().render())[G]
    widened = {}  # temporary -> h it holds
    seen = {g: [] for g in range(G)}
    for line in ins:
        m = re.match(r"v_(lshlrev|and)_b32 %\[(t\d)\], \S+ %\[x(\d)_(\d)\]", line)
        if m:
            dword = int(m.group(3)) * 4 + int(m.group(4))
            widened[m.group(2)] = 2 * dword + (0 if m.group(1) == "lshlrev" else 1)
            continue
        m = re.match(r"v_fmac_f32_dpp %\[a(\d)\], %\[w(\d)_(\d)\], %\[(t\d)\] row_newbcast:(\d+)", line)
        if m:
            g, wg, c, t, j = int(m.group(1)), int(m.group(2)), int(m.group(3)), m.group(4), int(m.group(5))
            assert wg == g
            h = 4 * j + c
            assert widened[t] == h, (line, widened[t], h)
            seen[g].append(h)
    for g in range(G):
        assert seen[g] == list(range(64))
