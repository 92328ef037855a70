"""Closed-form sizes the paper prints (test infrastructure).

* Appendix D: per-layer compactor parameter count
    p_l = H t d_l + B_c (2 n_c d_l^2 + 4 d n_c d_l) + B (4 n_s d_l^2)
          + B (2 r d_l^2) + (2 d_l d + d_l)
  (latent bank, cross-attention, self-attention, FFN if enabled, output heads
  including the optional beta head; small biases ignored).
* Appendix B, deployment accounting: KV bytes M_KV(S) = 2 L H_kv d b S.
"""


def compactor_params_per_layer(H, t, d, d_l, B, B_c, n_c, n_s, r, ffn=True, self_attn=True):
    p = H * t * d_l
    p += B_c * (2 * n_c * d_l ** 2 + 4 * d * n_c * d_l)
    if self_attn:
        p += B * (4 * n_s * d_l ** 2)
    if ffn:
        p += B * (2 * r * d_l ** 2)
    p += 2 * d_l * d + d_l
    return p


def kv_bytes(L, H_kv, d, b, S):
    return 2 * L * H_kv * d * b * S
