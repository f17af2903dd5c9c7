"""Comparison rules between the HIP path and the CPU oracle.

Bit-exact: per-sequence error bits, accepted counts and emitted tokens of every
sequence whose decisions are not ties (the oracle flags a sequence when an
acceptance test lies within 1e-6 of u, or the drawn token's CDF boundary lies
within 1e-6 probability mass of u' * Z).  Tie sequences are counted and checked
only for validity (accepted drafts are a prefix of the drafted tokens, the rest
is padding).

Floating point: KLD and draft entropy within 1e-4 relative plus 1e-7 absolute.
The statistics pass computes each exponential in fp32, adds the two of one
bf16 word in fp32 and everything after that in fp64.  KL = A/S_p - log S_p +
log S_q then carries two kinds of error: relative errors e_p, e_q of the sums
become an absolute KL error of about |e_q - e_p| (a few 1e-9 with these sums),
and the fp32 rounding of the exponentials themselves, relative errors d_v
and f_v of 2^(a_t) and 2^(a_d), shifts the result by about E_p[f - d] (the
log-ratio the KL accumulator uses is that of the unrounded exponents), which
reaches several 1e-8 when one token holds most of p.  A CPU emulation of the
kernel's order of operations against the fp64 oracle gives at most 0.71 of
this tolerance on 7,793 near-identical row pairs at V = 4096 and 0.56 on
2,000 close-draft pairs at V = 32000 (fp32 running sums per thread reached
1.2).  The 1e-7 floor covers KL values so small that 1e-4 of them is below
that.
"""
import numpy as np

KLD_REL, KLD_ABS = 1e-4, 1e-7
ENT_REL, ENT_ABS = 1e-4, 1e-7
LSE_ABS = 2e-5


def run_verify(dsde, step, row_lse=True):
    import torch
    lse = torch.empty((max(step.N, 1), 2), dtype=torch.float64, device=step.target.device)[:step.N] \
        if row_lse else None
    out = dsde.verify(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                      step.u_acc, step.u_res, step.k_max, row_lse=lse, draft_entropy=True)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    if lse is not None:
        res["row_lse"] = lse.cpu().numpy()
    return res


def _decode(row):
    row = np.asarray(row)
    if row.dtype == np.uint16:
        return (row.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return row.astype(np.float64)


def _softmax(z, T):
    s = z / float(T)
    s = s - s.max()
    e = np.exp(s)
    return e / e.sum()


def emission_is_valid(got, host, b, pad_id=-1):
    """A tie sequence's outputs are one of the emissions the method allows: the
    accepted drafts are a prefix of the drafted tokens, and the drawn token has
    positive weight (up to fp32 rounding) in the draw the accepted count implies
    (residual of the first rejected pair, or p of the bonus row), then padding."""
    sl, cu = host["sl"], host["cu_sl"]
    s, first, V = int(sl[b]), int(cu[b]), int(host["V"])
    a = int(got["accepted"][b])
    toks = got["tokens"][b]
    if not 0 <= a <= s:
        return False
    if not np.array_equal(toks[:a], host["draft_tokens"][first:first + a]):
        return False
    if (toks[a + 1:] != pad_id).any():
        return False
    y = int(toks[a])
    if not 0 <= y < V:
        return False
    T = host["temperature"][b]
    p = _softmax(_decode(host["target"][first + b + a]), T)
    if a == s:
        return p[y] > 0
    q = _softmax(_decode(host["draft"][first + a]), T)
    w = np.maximum(p - q, 0.0)
    if w.sum() <= 1e-12:
        return p[y] > 0
    return p[y] - q[y] > -1e-6 * max(p[y], q[y], 1e-30) - 1e-12


def compare_verify(got, ref, sl, cu_sl, label="", host=None):
    """Asserts the comparison rules; returns a small report.  With the host
    inputs given, tie sequences are also checked to be valid emissions."""
    B = len(sl)
    err_g = got["seq_err"].astype(np.uint32)
    err_r = ref["seq_err"].astype(np.uint32)
    assert np.array_equal(err_g, err_r), f"{label}: error bits differ: {np.nonzero(err_g != err_r)[0][:10]}"
    fine = err_r == 0
    ties = (ref["acc_tie"] != 0) | (ref["cdf_tie"] != 0)
    cmp = fine & ~ties
    bad_acc = np.nonzero(cmp & (got["accepted"] != ref["accepted"]))[0]
    assert bad_acc.size == 0, f"{label}: accepted differs at {bad_acc[:10]}: " \
                              f"{got['accepted'][bad_acc[:5]]} vs {ref['accepted'][bad_acc[:5]]}"
    bad_tok = np.nonzero(cmp & (got["tokens"] != ref["tokens"]).any(axis=1))[0]
    assert bad_tok.size == 0, f"{label}: tokens differ at {bad_tok[:10]}"
    # tie sequences: outputs are still a valid emission
    for b in np.nonzero(fine & ties)[0]:
        a = int(got["accepted"][b])
        assert 0 <= a <= sl[b]
        toks = got["tokens"][b]
        assert (toks[a + 1:] == -1).all()
        if host is not None:
            assert emission_is_valid(got, host, b), f"{label}: tie sequence {b} emits an invalid draw"
    # errored sequences get the defined fallback
    for b in np.nonzero(~fine)[0]:
        assert got["accepted"][b] == 0 and (got["tokens"][b] == -1).all()
    # KLD
    N = int(cu_sl[-1]) if len(cu_sl) else 0
    pos_fine = np.repeat(fine, sl) if N == len(ref["kld"]) else np.zeros(len(ref["kld"]), bool)
    kg = got["kld"].astype(np.float64)
    kr = ref["kld"]
    if pos_fine.any():
        d = np.abs(kg[pos_fine] - kr[pos_fine])
        lim = KLD_REL * np.abs(kr[pos_fine]) + KLD_ABS
        worst = int(np.argmax(d - lim))
        assert (d <= lim).all(), f"{label}: kld off by {d[worst]:.3g} (ref {kr[pos_fine][worst]:.6g})"
    if "draft_entropy" in got and pos_fine.any():
        eg = got["draft_entropy"].astype(np.float64)[pos_fine]
        er = ref["entropy"][pos_fine]
        de = np.abs(eg - er)
        assert (de <= ENT_REL * np.abs(er) + ENT_ABS).all(), f"{label}: draft entropy off by {de.max():.3g}"
    report = {"B": B, "compared": int(cmp.sum()), "acc_ties": int((ref["acc_tie"] != 0).sum()),
              "cdf_ties": int((ref["cdf_tie"] != 0).sum()), "errored": int((~fine).sum())}
    if "row_lse" in got and pos_fine.any():
        dl = np.abs(got["row_lse"][pos_fine] - ref["lse"][pos_fine])
        report["lse_max_abs_err"] = float(dl.max())
        assert dl.max() <= LSE_ABS, f"{label}: row lse off by {dl.max():.3g}"
    if pos_fine.any():
        dk = np.abs(kg[pos_fine] - kr[pos_fine])
        report["kld_max_rel_err"] = float((dk / np.maximum(np.abs(kr[pos_fine]), 1e-12)).max())
        report["kld_max_abs_err"] = float(dk.max())
        report["kld_err_over_tol"] = float((dk / (KLD_REL * np.abs(kr[pos_fine]) + KLD_ABS)).max())
    return report
