"""CPU oracle for the AsymSpec decision step.

Test infrastructure only: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the product package.
"""
from .asymspec_ref import (DELTA_A, DELTA_AB, DELTA_TB, GATE_CDA, GATE_FIXED,
                           GATE_KL, GATE_LAMBDA, LN2, RequestResult, RowResult,
                           argmax_first, bf16_bits_to_f32, divergence, fuse_verify,
                           fuse_verify_xvocab, fused_logits_f32,
                           fused_logprobs_full, gamma_eff, inverse_cdf, jsd, kl,
                           map_to_verifier,
                           log_ratio_at, log_softmax, softmax, to_f32,
                           verify_request)
from .emitted_law import (acceptance_prob, chi_square_stat, emitted_law,
                          first_token_law, total_variation)
