"""The oracle's pins have power: each mistake below, planted in a temporary
copy of the oracle, makes its CPU pin tests fail.

Every planted mistake is a plausible slip in reading the paper or writing
the oracle (a tie broken the other way, a dropped renormalisation, an
unsquared ReLU, a transposed operand, a wrong gradient operand, a missing
term of Eq. 1, a wrong MX-FP8 rounding or scale rule, ...).  Each runs the
pin tests (tests/test_oracle_*.py) in a subprocess whose ``oracle`` package
is the mutated copy; the library and the GPU are not involved.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

ROOT = Path(__file__).resolve().parents[1]

# (name, text in oracle/moe_oracle.py, planted replacement)
MUTATIONS = [
    ('tie_high_index',
     'choice = np.argmax(cand, axis=1)',
     'choice = cand.shape[1]-1-np.argmax(cand[:, ::-1], axis=1)'),
    ('no_renorm',
     'p = sel / sel.sum(axis=1, keepdims=True)',
     'p = sel'),
    ('relu_not_squared',
     'h[a:b] = np.maximum(u[a:b], 0.0) ** 2',
     'h[a:b] = np.maximum(u[a:b], 0.0)'),
    ('transpose_w1',
     'u[a:b] = x_disp[a:b] @ w1',
     'u[a:b] = x_disp[a:b] @ w1.T'),
    ('slot_order',
     '            perm[pos] = t * K + k',
     '            perm[pos] = k * S + t'),
    ('combine_no_weight',
     'w = 1.0 if p_disp is None else np.asarray(p_disp, np.float64)[pos][:, None]\n        y = y + w',
     'w = 1.0\n        y = y + w'),
    ('drelu_factor',
     'du[a:b] = dh * (2.0 * np.maximum(u[a:b], 0.0))',
     'du[a:b] = dh * (np.maximum(u[a:b], 0.0))'),
    ('dw2_wrong',
     'dW2[e] = h[a:b].T @ dy_disp[a:b]',
     'dW2[e] = u[a:b].T @ dy_disp[a:b]'),
    ('eq1_no_bp',
     'return S * K * (D * b_x + b_p)',
     'return S * K * (D * b_x)'),
    ('nan_high',
     'v = np.where(num, vals, -np.inf)',
     'v = np.where(num, vals, -np.inf); num = avail'),
    ('bf16_trunc',
     'r = np.rint(v / ulp) * ulp',
     'r = np.trunc(v / ulp) * ulp'),
    ('hidden_not_rounded',
     '            h[a:b] = round_bf16(h[a:b])',
     '            h[a:b] = h[a:b]'),
    ('latent_combine_not_rounded',
     '        if round_activations:\n            y = round_bf16(y)',
     '        if round_activations:\n            y = y'),
    ('bias_ignored',
     'z = z + np.asarray(bias, np.float64)[None, :]',
     'z = z'),
    ('gates_from_biased',
     '    sel = np.take_along_axis(s, np.asarray(idx, np.int64), axis=1)\n    tot = sel.sum(axis=1, keepdims=True)\n    if np.any',
     '    s = s + 0.1 * np.arange(s.shape[1])[None, :]\n    sel = np.take_along_axis(s, np.asarray(idx, np.int64), axis=1)\n    tot = sel.sum(axis=1, keepdims=True)\n    if np.any'),
    ('sel_tie_high',
     'order = np.lexsort((experts, -key[t]))',
     'order = np.lexsort((-experts, -key[t]))'),
    ('sel_ignores_bias',
     'key = s if sel_bias is None else s + np.asarray(sel_bias, np.float64)[None, :]',
     'key = s'),
    ('aux_batch_level',
     '    B = _sequences(S, seq_len)\n    sn = s / s.sum(axis=1, keepdims=True)\n    total = 0.0\n    for b in range(B):\n        rows = slice(b * seq_len, (b + 1) * seq_len)',
     '    B = _sequences(S, seq_len)\n    sn = s / s.sum(axis=1, keepdims=True)\n    total = 0.0\n    seq_len = S; B_ = B; B = 1\n    for b in range(1):\n        rows = slice(0, S)'),
    ('aux_unnormalised',
     '    sn = s / s.sum(axis=1, keepdims=True)\n    total = 0.0',
     '    sn = s\n    total = 0.0'),
    ('aux_no_E_over_K',
     '        f = np.bincount(idx[rows].ravel(), minlength=E) * (E / (K * seq_len))\n        P = sn',
     '        f = np.bincount(idx[rows].ravel(), minlength=E) * (1 / seq_len)\n        P = sn'),
    ('auxbwd_no_center',
     '    ds = (a - np.sum(a * sn, axis=1, keepdims=True)) / tot',
     '    ds = a / tot'),
    ('gatebwd_no_sig_deriv',
     '            out[t, e] = dsel[t, k] * s[t, e] * (1.0 - s[t, e])',
     '            out[t, e] = dsel[t, k]'),
    ('shared_relu_plain',
     '    h = np.maximum(u, 0.0) ** 2\n    return u, h, h @',
     '    h = np.maximum(u, 0.0)\n    return u, h, h @'),
    ('shared_bwd_dws2',
     'return du @ Ws1.T, x.T @ du, np.asarray(h, np.float64).T @ dy',
     'return du @ Ws1.T, x.T @ du, np.asarray(u, np.float64).T @ dy'),
    ('bias_update_sign',
     'rate * np.sign(c.mean() - c)',
     'rate * np.sign(c - c.mean())'),
    ('layer_no_aux_grad',
     '            ds = ds + seq_aux_loss_bwd(fwd["logits"], fwd["topk_idx"], seq_len, aux_coeff)',
     '            pass'),
    ('layer_shared_dx_missing',
     '        dx_r = dx_r + dx_shared',
     '        dx_r = dx_r'),
    ('ties_away',
     '        r = np.rint(a[n] / ulp) * ulp        # may carry into the next binade',
     '        r = np.floor(a[n] / ulp + 0.5) * ulp'),
    ('emax_7',
     '    s = np.where(amax > 0, ex - 1 - E4M3_EMAX, -E8M0_BIAS)',
     '    s = np.where(amax > 0, ex - 1 - 7, -E8M0_BIAS)'),
    ('sat_480',
     '    a = np.minimum(np.abs(v), E4M3_MAX)',
     '    a = np.minimum(np.abs(v), 480.0)'),
    ('sub_step',
     '    code[sub] = np.rint(a[sub] / 2.0 ** -9).astype(np.int64)',
     '    code[sub] = np.rint(a[sub] / 2.0 ** -8).astype(np.int64)'),
    ('block16',
     'MX_BLOCK = 32\n',
     'MX_BLOCK = 16\n'),
    ('decode_bias8',
     '    val = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.ldexp(1.0, e - 7))',
     '    val = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.ldexp(1.0, e - 8))'),
    ('no_clamp_low',
     '    return np.clip(s, -E8M0_BIAS, E8M0_BIAS).astype(np.int64)',
     '    return np.clip(s, -200, E8M0_BIAS).astype(np.int64)'),
    ('payload_no_scale',
     '    return S * K * (D + D // MX_BLOCK + b_p)',
     '    return S * K * (D + b_p)'),
    ('sign_lost',
     '    sign = np.signbit(v).astype(np.uint8) << 7',
     '    sign = (v < 0).astype(np.uint8) << 7'),
    ('layer_no_quant',
     '        x_disp = mxfp8_dequantize(xq, xs)',
     '        x_disp = x_r'),
]


def _run(tmp: Path, name: str, old: str, new: str) -> int:
    d = tmp / name
    (d / "oracle").mkdir(parents=True)
    (d / "oracle" / "__init__.py").write_text((ROOT / "oracle" / "__init__.py").read_text())
    src = (ROOT / "oracle" / "moe_oracle.py").read_text()
    (d / "oracle" / "moe_oracle.py").write_text(src.replace(old, new, 1))
    shutil.copytree(ROOT / "tests", d / "tests",
                    ignore=shutil.ignore_patterns("__pycache__", "test_oracle_mutations.py"))
    os.symlink(ROOT / "paper_2608_28511_amd", d / "paper_2608_28511_amd")
    tests = sorted(str(p) for p in (d / "tests").glob("test_oracle_*.py"))
    r = subprocess.run([sys.executable, "-m", "pytest", *tests, "-q", "-x", "-p", "no:cacheprovider"],
                       cwd=d, capture_output=True, text=True, timeout=600)
    return r.returncode


def test_every_planted_mistake_is_caught(tmp_path):
    src = (ROOT / "oracle" / "moe_oracle.py").read_text()
    for name, old, _ in MUTATIONS:
        assert src.count(old) == 1, f"mutation site of {name} no longer in the oracle"
    # control: the same harness on the unmodified oracle passes
    assert _run(tmp_path, "unmodified", "", "") == 0
    with ThreadPoolExecutor(max_workers=4) as ex:
        codes = list(ex.map(lambda m: _run(tmp_path, *m), MUTATIONS))
    missed = [m[0] for m, c in zip(MUTATIONS, codes) if c == 0]
    assert not missed, f"planted mistakes not caught by the pins: {missed}"
    # every run failed on a test, not on a collection or usage error
    assert all(c == 1 for c in codes), dict(zip([m[0] for m in MUTATIONS], codes))
