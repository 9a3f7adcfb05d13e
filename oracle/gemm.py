"""The GEMM of Section 4 (C = A B) and its closed-formula tiles, as plain code.

Test infrastructure only: only tests/, the smoke check and the benchmark's CPU
leg may import this module, and it shares no code with the GPU library.

``gemm`` is the definition in float64.  ``derive`` applies the CU-centric
rules of Section 4 to a GEMM (the worked example of the section):

1. LDS -> CU tile.  The A and B tiles of one stage, (t_M + t_N) t_K elements,
   share LDS with the other stages; with t_M = t_N the square tile is
   floor(sqrt(LDS / elem)) and t_K = floor(LDS / (stages (t_M + t_N) elem)).
   (Reading: the printed closed form puts LDS/2 under the square root, which
   does not give the section's own numbers; sqrt(LDS/elem) with two stages
   does: 128, 128, 32 for 64 KB and 4-byte elements.)  t_M, t_N are aligned
   down to the atom times the waves along each dimension, t_K to the atom's k.
2. VGPR -> warp tile.  Each wave accumulates a (t_M / waves_m) x (t_N /
   waves_n) block of C: (t_wm / m)(t_wn / n) atoms of m n acc_bytes /
   (4 wavefront) registers each, plus a fixed overhead, within the budget at
   the kernel's waves per SIMD; the CU tile halves (the larger side first)
   until it fits.
3. CU count -> grid.  ceil(M / t_M) ceil(N / t_N) workgroups; while that is
   below the CU count the larger tile side halves, down to one atom per wave.
4. Atom alignment throughout, and t_K also such that each of the A and B
   tiles of a stage is a whole number of copy blocks per wave (a structure
   property: every wave moves the same number of copy_block-byte blocks).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


def gemm(a, b):
    """C = A B in float64."""
    return np.asarray(a, dtype=np.float64) @ np.asarray(b, dtype=np.float64)


@dataclasses.dataclass(frozen=True)
class GemmStructure:
    """Fixed properties of one GEMM kernel family."""
    stages: int = 2          # A+B tile stages resident in LDS
    waves_m: int = 2         # wave grid over the CU tile
    waves_n: int = 2
    waves_per_simd: int = 1
    vgpr_fixed: int = 32
    copy_block: int = 0      # bytes one wave moves per copy instruction (0: no constraint)


def derive(lds_bytes, vgpr_per_thread, wavefront_size, num_cus, atom_m, atom_n, atom_k, elem, acc_bytes,
           M, N, K, st: GemmStructure = GemmStructure()):
    """Returns a dict of tiles and the binding constraint, or None if even one
    atom per wave does not fit."""
    am, an = atom_m * st.waves_m, atom_n * st.waves_n
    t = int(math.isqrt(lds_bytes // elem))
    t_m = t // am * am
    t_n = t // an * an
    if t_m < am or t_n < an:
        return None

    def t_k_of(tm, tn):
        step = atom_k
        if st.copy_block:
            unit = st.copy_block * st.waves_m * st.waves_n
            for side in (tm, tn):
                need = unit // math.gcd(unit, side * elem)
                step = step * need // math.gcd(step, need)
        return lds_bytes // (st.stages * (tm + tn) * elem) // step * step

    budget = vgpr_per_thread // st.waves_per_simd

    def regs(tm, tn):
        wm, wn = tm // st.waves_m, tn // st.waves_n
        per_atom = -(-(atom_m * atom_n * acc_bytes) // (4 * wavefront_size))
        return (wm // atom_m) * (wn // atom_n) * per_atom + st.vgpr_fixed

    binding = "LDS"
    while regs(t_m, t_n) > budget:
        if t_m >= t_n and t_m > am:
            t_m = max(am, t_m // 2 // am * am)
        elif t_n > an:
            t_n = max(an, t_n // 2 // an * an)
        else:
            return None
        binding = "VGPR"
    while -(-M // t_m) * -(-N // t_n) < num_cus and (t_m > am or t_n > an):
        if (t_m >= t_n and t_m > am) or t_n <= an:
            t_m = max(am, t_m // 2 // am * am)
        else:
            t_n = max(an, t_n // 2 // an * an)
        binding = "CU"
    t_k = t_k_of(t_m, t_n)
    if t_k < atom_k:
        return None
    grid = -(-M // t_m) * -(-N // t_n)
    return dict(t_m=t_m, t_n=t_n, t_k=t_k, warp_m=t_m // st.waves_m, warp_n=t_n // st.waves_n, grid=grid,
                vgpr_est=regs(t_m, t_n), vgpr_budget=budget, lds_used=st.stages * (t_m + t_n) * t_k * elem,
                wg_per_cu=grid / num_cus, binding=binding)
