"""Plain, slow CPU oracle of the KV-COBRA hot path.

THIS PACKAGE IS TEST INFRASTRUCTURE. Only tests/, the smoke check in
__graft_entry__.py and the cpu_baseline leg of bench.py may import, call,
link or run anything under oracle/. The GPU library and its Python binding
never import it, and the oracle never imports them; the two share no code.

Modules
-------
quant      quantizer, distortion model q(b), per-head step (Eq. eq:q, Appendix A.1)
alloc      C1, C2 damped update, exact DP, brute force (Sections 3.2-3.3, 4; Appendices B-D, F)
basis      fused Hadamard-rotated basis and step (Section 3.4; table steps 5-6)
layout     packed code-stream layout, pure Python (tiny inputs)
native     exact encode, pack, unpack in C (kvc_oracle.c), for realistic sizes
attention  dequantize, reconstruct, decode attention and dense softmax attention in fp64

Parity status: every function here is pinned by tests in tests/test_oracle_*.py
against closed forms, invariants, brute force or exact rational arithmetic,
except the damped C2 allocation, whose agreement with a global optimum the
paper does not claim ("parity unpinned" for optimality; only its invariants
and the Table steps are checked).
"""
