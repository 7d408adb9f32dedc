"""GPU parity of the benchmarked step itself: the workload's whole stack run by
``paper_2608_01653_amd.stack.Stack.step`` (the composition ``bench.py`` times,
at the benchmark's full size and launch configuration), checked sample by
sample against the oracle, teacher-forced layer by layer (Table I, Fig.
hadamard_framework): each oracle stage consumes the GPU's previous outputs for
that sample, so every stage is compared on identical inputs.

Per-sample scales make samples independent, so a few samples of the batch
stand for the rest.  Rules per stage:
* the first layer's codes (WH: no transform): bit-exact, scale bit-exact;
* layer 1 -> 2 (WH 64 -> DH 64, both transforms explicit): codes of the
  oracle's composition fl32(B_next y_ref) under the code rule, the scale within
  the bound of the GPU's fp32 butterflies;
* DH convolutions: fp32 output bit-exact; the fused next-operand absmax equal
  to the two-pass activation kernel's on the stored output and within the
  fp32-butterfly bound of the oracle's;
* DH activation passes: code rule, scale within the bound; WH activation
  passes (no transform): bit-exact;
* the last (WH) convolution: range-relative 1e-6.
"""
import numpy as np
import pytest
import torch

from gpu_util import assert_codes, assert_range_rel, assert_scale_ulp, host
from paper_2608_01653_amd import hatq, stack, workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    hatq.load()
    torch.cuda.init()


def _gamma(k):
    u = 2.0 ** -24
    return k * u / (1 - k * u)


def _stages(b):
    """Rounded fp32 stages between a value and its transform: log2(b) for a
    Sylvester block; the 16-point butterfly then the Paley factor's b/16 - 1
    sums for the Kronecker orders."""
    return 4 + b // 16 - 1 if b in (192, 320) else int(np.log2(b)) if b > 1 else 0


def _butterfly_absmax_tol(y, b):
    """|max|B y|_fp32-butterfly - max|fl32(B y)|_fp64| bound for one sample: each
    value differs by at most gamma_stages(b) * (sum of |y| over its block) plus
    the oracle's own rounding."""
    if b == 1:
        return 0.0
    ya = np.abs(y.astype(np.float64)).reshape(-1, b).sum(-1).max()
    return _gamma(_stages(b)) * ya + 2.0 ** -24 * np.abs(y).max() * b


def _oracle_prepared(orc, wl, params):
    out = []
    for L, (w, b) in zip(wl.layers, params):
        out.append(orc.prepare_weights(w, b, cin=L.cin, cout=L.cout, k=L.k, stride=L.stride, pad=L.pad,
                                       form=L.form, hblock=L.hblock, transposed=L.transposed, out_pad=L.out_pad))
    return out


def _conv(orc, xq, pw):
    return orc.conv_int8(xq, pw.wq, stride=pw.stride, pad=pw.pad, transposed=pw.transposed, out_pad=pw.out_pad)


def _check_sample(orc, st, refs, x0, s, paired):
    wl = st.wl
    sl = slice(s, s + 1)
    g = lambda t: host(t[sl])                                          # noqa: E731
    # layer 1 activation pass (WH: original domain)
    q_ref, s_ref = orc.quantize_symmetric(orc.activation_transform(x0[sl], st.act_hb[0]))
    assert np.array_equal(g(st.sc[0]), s_ref)
    assert_codes(g(st.codes(0)), q_ref, exact=True, what=f"sample {s} layer 1 codes")
    for i in range(st.nL):
        pw = refs[i]
        xq_i, sx_i = g(st.codes(i)), g(st.sc[i])
        acc = _conv(orc, xq_i, pw)
        y_ref = orc.epilogue(acc, sx_i, pw)
        if i + 1 == st.nL:
            (np.testing.assert_array_equal if pw.form == "DH" else assert_range_rel)(g(st.ys[i]), y_ref)
            break
        nb = st.act_hb[i + 1]
        if st.requant[i]:
            # the next operand's codes straight from the epilogue
            S = orc.activation_transform(y_ref, nb)
            q_ref, s_ref = orc.quantize_symmetric(S)
            tol = _butterfly_absmax_tol(y_ref, nb)
            if pw.form == "WH":
                za = np.abs(orc.wh_z(acc, sx_i, pw).astype(np.float64))
                hb = pw.hblock
                dy = _gamma(_stages(hb)) * za.reshape(-1, hb).sum(-1).max() / hb
                tol += max(nb, 1) * (dy + 2.0 ** -24 * np.abs(y_ref).max())
            s_tol = tol / 127 + 2 * np.spacing(np.float32(s_ref[0]))
            assert abs(float(g(st.sc[i + 1])[0]) - float(s_ref[0])) <= s_tol
            assert_codes(g(st.codes(i + 1)), q_ref, what=f"sample {s} layer {i + 1} -> {i + 2} codes"
                         + (" (paired)" if paired else ""))
            continue
        y_gpu = g(st.ys[i])
        if pw.form == "DH":
            np.testing.assert_array_equal(y_gpu, y_ref)
        else:
            assert_range_rel(y_gpu, y_ref)
        # the next layer's fused absmax against the oracle's transform of the GPU output
        S = orc.activation_transform(y_gpu, nb)
        A_ref = float(np.abs(S.astype(np.float64)).max())
        assert abs(float(g(st.amax[i])[0]) - A_ref) <= _butterfly_absmax_tol(y_gpu, nb)
        q_ref, s_ref = orc.quantize_symmetric(S)
        if nb == 1:
            assert np.array_equal(g(st.sc[i + 1]), s_ref)
            assert_codes(g(st.codes(i + 1)), q_ref, exact=True, what=f"sample {s} layer {i + 2} codes")
        else:
            s_tol = _butterfly_absmax_tol(y_gpu, nb) / 127 + 2 * np.spacing(np.float32(s_ref[0]))
            assert abs(float(g(st.sc[i + 1])[0]) - float(s_ref[0])) <= s_tol
            assert_codes(g(st.codes(i + 1)), q_ref, what=f"sample {s} layer {i + 2} codes")


@pytest.mark.parametrize("name,samples", [("analysis_stack4_rgb_512x768", [0]),
                                          ("analysis_stack4_rgb_b16_1024x1024", [0, 15])])
@pytest.mark.parametrize("paired", [False, True])
def test_stack_step_teacher_forced(orc, name, samples, paired):
    wl = workloads.ALL[name]
    x_np, params = wl.generate()
    st = stack.Stack(wl, params)
    x0 = torch.from_numpy(x_np).to(st.dev)
    st.step(x0, paired=paired)
    torch.cuda.synchronize()
    # fused absmax = what the two-pass activation kernel computes from the stored outputs
    for i in range(st.nL - 1):
        if not st.requant[i]:
            q1, s1 = hatq.hatq_fwht_quant_act(st.ys[i], st.act_hb[i + 1])
            assert torch.equal(s1, st.sc[i + 1]) and torch.equal(q1, st.codes(i + 1))
            del q1
    refs = _oracle_prepared(orc, wl, params)
    for s in samples:
        _check_sample(orc, st, refs, x_np, s, paired)


@pytest.mark.parametrize("name,samples", [("analysis_stack4_rgb_512x768", [0]),
                                          ("analysis_stack4_rgb_b16_1024x1024", [0, 15])])
def test_stack_paper_orders_teacher_forced(orc, name, samples):
    """The stack with one block of the paper's order m(C) per transformed axis
    (Eq. hadamard_order: 192, 192, 192, 320) instead of blocks of 64: the WH
    restore of order 192 and the next operand's order 192 in layer 1's two
    passes, order 192 in the quantizer and in the fused absmax, and the order-320
    WH restore of layer 4 on the 320-column tile; same rules per stage (at the
    batch-16 size, the step the bench's paper-order leg times)."""
    wl = workloads.with_orders(workloads.ALL[name], hatq.hatq_hadamard_order)
    assert [L.hblock for L in wl.layers] == [192, 192, 192, 320]
    x_np, params = wl.generate()
    st = stack.Stack(wl, params)
    x0 = torch.from_numpy(x_np).to(st.dev)
    st.step(x0)
    torch.cuda.synchronize()
    for i in range(st.nL - 1):
        if not st.requant[i]:
            q1, s1 = hatq.hatq_fwht_quant_act(st.ys[i], st.act_hb[i + 1])
            assert torch.equal(s1, st.sc[i + 1]) and torch.equal(q1, st.codes(i + 1))
    refs = _oracle_prepared(orc, wl, params)
    for s in samples:
        _check_sample(orc, st, refs, x_np, s, False)
