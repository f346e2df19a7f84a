"""CPU float64 oracle for the SAKI coupling-and-routing path.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain, obviously
correct statement of what the HIP library computes.  Only the test suite,
the smoke check and the bench's CPU-baseline leg may import it; the product
path (the C-ABI library and its Python binding) never imports, calls or
links anything here, and shares no code with it.

Modules
-------
philox    Philox-4x32-10 (Salmon et al., SC'11) and the stream layout.
bridge    log-softmax, the geometric bridge q_lambda, KL(q||p), the
          trust-region coefficient lambda*, TV(p, q)   (Sec. 3.2, App. A).
coupling  maximal coupling: proposal race, accept test, residual race
          (Sec. 3.3, Eq. accept / Eq. residual, App. D).
routing   routed loss and its gradient (Sec. 3.4, Eq. general_objective,
          App. B, App. H).
verify    speculative block verification with first-rejection semantics
          (Sec. 3.5, App. F, App. I).
supervision  teacher-sampled correction targets (App. C) and the Random-TM /
          TV-Weighted-TM placement controls (Sec. 4.1, placement-control
          appendix).
probe     fixed-prefix probe metrics C_1, C_k, KL(T || S), H(S).
rollout   multi-wave speculative rollout: drafting, verification,
          first-rejection commit and rollback, token-aligned metadata
          (Sec. 3.5, App. F Prop. spec_exact, App. I).

Every function works in float64 on the exact input values (bf16 and fp32
logits convert exactly to float64).
"""
