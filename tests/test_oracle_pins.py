"""The CPU oracle against what the paper and the mathematics fix (no GPU)."""
import importlib.util
import os

import pytest

import oracle.msa_oracle as O
from tests import pins

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                          "oracle", "msa_oracle.py")


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(O)


# Plausible mistakes planted in a copy of the oracle; each must trip a pin.
MUTATIONS = {
    "rank_ascending": ("order = np.lexsort((cand, -m_rank[:lb].astype(np.float64)))",
                       "order = np.lexsort((cand, m_rank[:lb].astype(np.float64)))"),
    "tie_higher_id": ("order = np.lexsort((cand, -m_rank[:lb].astype(np.float64)))",
                      "order = np.lexsort((-cand, -m_rank[:lb].astype(np.float64)))"),
    "local_not_reserved": ("others = topk - 1                          # one slot",
                           "others = topk                              # one slot"),
    "causal_cut_off_by_one": ("vis = dots_row[:pos + 1]", "vis = dots_row[:pos]"),
    "own_token_dropped": ("np.arange(b * block_size, min((b + 1) * block_size, pos + 1))",
                          "np.arange(b * block_size, min((b + 1) * block_size, pos))"),
    "no_softmax_scale": ("z = (qh @ keys.T) * scale", "z = (qh @ keys.T)"),
    "lse_log2": ("lse = (m + np.log(l))[:, 0]", "lse = (m + np.log2(l))[:, 0]"),
    "combine_weight_sign": ("w = np.exp(lse_parts - lse)", "w = np.exp(lse - lse_parts)"),
    "flops_main_factor": ("4.0 * H_q * d_h * N * k * block_size", "2.0 * H_q * d_h * N * k * block_size"),
    "left_aligned_positions": ("return s, self.kv_lens[s] - self.q_rows[s] + t", "return s, t"),
    "fp8_exponent_bias": ("np.ldexp(1.0 + m / 8.0, e - 7)", "np.ldexp(1.0 + m / 8.0, e - 8)"),
    "fp8_subnormal_scale": ("np.ldexp(m / 8.0, -6)", "np.ldexp(m / 8.0, -7)"),
    "fp8_nan_all_top_exponent": ("v = np.where((e == 15) & ((c & 0x7) == 7), np.nan, v)",
                                 "v = np.where(e == 15, np.nan, v)"),
    "fp8_v_scale_dropped": ("vals = dec(v_bits[kv0 + toks, g]) * vs", "vals = dec(v_bits[kv0 + toks, g])"),
    "bwd_softmax_jacobian_no_mean": ("dz = p * (dp - (p * dp).sum(axis=1, keepdims=True))", "dz = p * dp"),
    "bwd_dk_unscaled": ("dk = (dz.T @ qh) * scale", "dk = (dz.T @ qh)"),
    "bwd_dv_scaled": ("dv = p.T @ d_o", "dv = (p.T @ d_o) * scale"),
    "bwd_dk_into_group0": ("dK[kv0 + toks, g] += dk", "dK[kv0 + toks, 0] += dk"),
    "kl_teacher_logit_mean": ("p = softmax_rows((q_heads @ k_toks.T) * scale_main).mean(axis=0)",
                              "p = softmax_rows(((q_heads @ k_toks.T) * scale_main).mean(axis=0)[None, :])[0]"),
    "kl_grad_sign": ("ds = p_idx - p", "ds = p - p_idx"),
    "kl_reverse_direction": ("kl = float(np.sum(p * (np.log(p) - np.log(p_idx))))",
                             "kl = float(np.sum(p_idx * (np.log(p_idx) - np.log(p))))"),
    "kl_dq_unscaled": ("d_iq = (ds @ ik_toks) * scale_idx", "d_iq = (ds @ ik_toks)"),
    "tie_rule_dominance_flipped": (
        "return min(block_scores[b] for b in nonlocal_sel) >= max(block_scores[b] for b in unsel) - tol",
        "return max(block_scores[b] for b in unsel) >= min(block_scores[b] for b in nonlocal_sel) - tol"),
    "tie_rule_tolerance_sign": (
        "return min(block_scores[b] for b in nonlocal_sel) >= max(block_scores[b] for b in unsel) - tol",
        "return min(block_scores[b] for b in nonlocal_sel) >= max(block_scores[b] for b in unsel) + tol"),
    "tie_rule_local_not_checked": ("len(sel) != min(topk, lb + 1) or lb not in sel:",
                                   "len(sel) != min(topk, lb + 1):"),
    "tie_rule_padding_not_checked": ("or any(int(b) != -1 for b in ids[len(sel):])", "or False"),
    "tie_rule_order_not_checked": ("if list(ids[:len(sel)]) != sorted(sel) or", "if"),
    "tie_rule_past_local_allowed": ("if any(b < 0 or b > lb for b in sel):", "if any(b < 0 for b in sel):"),
    "row_scores_unscaled": ("return block_maxima(d, pos, block_size) / math.sqrt(iq.shape[0])",
                            "return block_maxima(d, pos, block_size)"),
    "row_scores_causal_cut": ("ik = decode_bf16(index_k_bits[kv0:kv0 + pos + 1])\n    iq = decode_bf16(index_q_bits[row, group])",
                              "ik = decode_bf16(index_k_bits[kv0:kv0 + pos])\n    iq = decode_bf16(index_q_bits[row, group])"),
    "row_scores_no_kv_start": ("ik = decode_bf16(index_k_bits[kv0:kv0 + pos + 1])\n    iq = decode_bf16(index_q_bits[row, group])",
                               "ik = decode_bf16(index_k_bits[0:pos + 1])\n    iq = decode_bf16(index_q_bits[row, group])"),
    "row_topk_smallest": ("order = np.lexsort((cols, -scores[i].astype(np.float64)))",
                          "order = np.lexsort((cols, scores[i].astype(np.float64)))"),
    "row_topk_tie_higher_column": ("order = np.lexsort((cols, -scores[i].astype(np.float64)))",
                                   "order = np.lexsort((-cols, -scores[i].astype(np.float64)))"),
    "row_topk_rank_order_output": ("sel = np.sort(cols[order[:k]])", "sel = cols[order[:k]]"),
    "row_topk_one_short": ("sel = np.sort(cols[order[:k]])", "sel = np.sort(cols[order[:k - 1]])"),
    "head_to_group_modulo": ("O[i, g * G:(g + 1) * G], L[i, g * G:(g + 1) * G] = attend(\n                qf[g * G:(g + 1) * G], keys, vals, scale)",
                             "O[i, g::H_kv], L[i, g::H_kv] = attend(\n                qf[g::H_kv], keys, vals, scale)"),
}


def _mutant(name, old, new):
    src = open(ORACLE_SRC).read()
    assert src.count(old) >= 1, f"mutation {name} does not apply"
    src = src.replace(old, new)
    spec = importlib.util.spec_from_loader(f"oracle_mutant_{name}", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src, f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_oracle_mutations_are_caught(name):
    old, new = MUTATIONS[name]
    mod = _mutant(name, old, new)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"no pin catches mutation {name}"
