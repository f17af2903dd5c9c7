"""Small host-side helpers shared by the tests (no arithmetic of the method)."""
import numpy as np


def bf16_bits(x):
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(x)
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def packed_layout(sls):
    """cu_sl (exclusive prefix sums) of a list of speculation lengths."""
    sl = np.asarray(sls, dtype=np.int32)
    cu = np.zeros(len(sl) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(sl)
    return sl, cu


def single_pair_batch(p_logits, q_logits, xs, us, u_res, temperature=1.0, bonus_logits=None):
    """A batch of B = len(xs) one-position sequences sharing one (target, draft)
    row pair: sequence i drafts token xs[i] with acceptance uniform us[i] and
    draw uniform u_res[i].  Returns the keyword arguments of ``oracle.verify``."""
    p_logits = np.asarray(p_logits, np.float32)
    q_logits = np.asarray(q_logits, np.float32)
    V = p_logits.shape[0]
    B = len(xs)
    bonus = p_logits if bonus_logits is None else np.asarray(bonus_logits, np.float32)
    target = np.empty((2 * B, V), np.float32)
    target[0::2] = p_logits
    target[1::2] = bonus
    draft = np.broadcast_to(q_logits, (B, V)).copy()
    sl, cu = packed_layout([1] * B)
    return dict(target=target, draft=draft, V=V, sl=sl, cu_sl=cu,
                draft_tokens=np.asarray(xs, np.int32),
                temperature=np.full(B, temperature, np.float32),
                u_acc=np.asarray(us, np.float32), u_res=np.asarray(u_res, np.float32), k_max=1)
