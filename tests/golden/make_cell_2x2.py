"""Derive the values of cell_2x2.txt: hand-worked 2x2 MDLSTM grids, one hidden
unit, one input channel, every cell written out with scalar math and its own
predecessor table per scan direction (independent of ``oracle/``).

The cell is the two-predecessor MDLSTM cell of Section III (two forget gates
weighing the two predecessor states); the gate biases are chosen so that the
four sigmoid gates take exact values (3/4, 1/4, 1/2, 4/5) and only the cell
candidate depends on the input and the predecessors' hidden states.
Predecessors outside the grid hand over zeros (Section V, masking).

Usage: python tests/golden/make_cell_2x2.py   (prints the derivation; the
RESULT lines are the fixture's h and c values, row-major per direction)
"""
from math import exp, log, tanh


def sig(z):
    return 1.0 / (1.0 + exp(-z))


X = {(0, 0): 0.0, (0, 1): 1.0, (1, 0): 2.0, (1, 1): 3.0}
WG, BG, UL, UT = 0.5, 0.25, 1.0, -2.0          # candidate: a_g = WG x + BG + UL h_L + UT h_T
I, FL, FT, O = 0.75, 0.25, 0.5, 0.8            # sig(ln 3), sig(-ln 3), sig(0), sig(ln 4)
assert abs(sig(log(3)) - I) < 1e-15 and abs(sig(-log(3)) - FL) < 1e-15
assert abs(sig(0.0) - FT) < 1e-15 and abs(sig(log(4)) - O) < 1e-15


def cell(p, left, top, state):
    hl, cl = state.get(left, (0.0, 0.0))
    ht, ct = state.get(top, (0.0, 0.0))
    ag = WG * X[p] + BG + UL * hl + UT * ht
    g = tanh(ag)
    c = I * g + FL * cl + FT * ct
    h = O * tanh(c)
    state[p] = (h, c)
    print(f"  cell {p}: L={left} T={top} hL={hl:.15f} hT={ht:.15f} cL={cl:.15f} cT={ct:.15f}")
    print(f"     a_g={ag:.15f} g={g:.15f} c={c:.15f} h={h:.15f}")


# scan order and predecessor offsets of each direction, written out
DIRECTIONS = [
    ([(0, 0), (0, 1), (1, 0), (1, 1)], lambda y, x: (y, x - 1), lambda y, x: (y - 1, x)),  # from top-left
    ([(0, 1), (0, 0), (1, 1), (1, 0)], lambda y, x: (y, x + 1), lambda y, x: (y - 1, x)),  # from top-right
    ([(1, 0), (1, 1), (0, 0), (0, 1)], lambda y, x: (y, x - 1), lambda y, x: (y + 1, x)),  # from bottom-left
    ([(1, 1), (1, 0), (0, 1), (0, 0)], lambda y, x: (y, x + 1), lambda y, x: (y + 1, x)),  # from bottom-right
]

if __name__ == "__main__":
    for d, (order, left_of, top_of) in enumerate(DIRECTIONS):
        print(f"direction {d}")
        st = {}
        for p in order:
            cell(p, left_of(*p), top_of(*p), st)
        print("RESULT", d, " ".join(f"{st[(y, x)][0]:.15e} {st[(y, x)][1]:.15e}" for y in (0, 1) for x in (0, 1)))
