"""Helpers shared by the GPU parity tests: upload the seeded inputs, run the
library through its C ABI, run the oracle on the same bytes, and compare.

The parity bar (``check``), element by element:

  bf16 outputs   |got - ref| <= 2e-2 + u(max(|got|, |ref|)) + A + C
  fp32 outputs   relative Frobenius and per-row only, unless an absolute
                 bound is given: |got - ref| <= abs_bound + A

u(r) is the spacing of the bf16 grid at |r|.  2e-2 is the stated max-abs
tolerance; u admits the output's own rounding (two fp32 values that differ in
the last bits can round to neighbouring bf16 values, so 2e-2 alone is below
bf16 resolution for |x| >= 4), taken at the larger magnitude because a value
next to a power of two can round into the binade above.

A (flip allowance) is zero unless a test passes it.  It is computed per
element from the oracle's values of the stored bf16 operands that feed that
element directly (elementwise): for each such operand o, |d out / d o| u(o), the
change one rounding flip of o makes (o rounds one step to the neighbouring
bf16 value where its fp32 sum lands next to a rounding boundary).
``layer_allowances`` lists them for the layer.

C (contraction allowance) applies to outputs computed by a contraction (a
GEMM or attention) from operands that carry errors of their own: C = 6 x 5e-3
x RMS of the reference over the element's row.  If the operands deviate from
the oracle by the stated relative tolerance 5e-3 with independent errors, an
output element of a contraction deviates by about 5e-3 times the RMS of its
row (for y = a W, the error of y_i is sum_j e_j W_ji, of standard deviation
5e-3 |a| |W_i| ~ 5e-3 RMS(y)), whatever the element's own magnitude, which
cancellation can make small; 6 standard deviations cover the largest of the
10^7 - 10^8 elements of a full-size tensor.  Elementwise outputs (the RMSNorm
outputs, act, prod) get no C of their own; their A carries the bounds of the
contraction outputs they are computed from.

On top of the element bound, every float output must meet
  * relative Frobenius error <= 5e-3 over the tensor (stated), and
  * relative error <= 2e-2 on every row (last axis; floor: 2e-2 of the
    tensor's RMS row norm), so that one wrong row cannot hide in a large
    tensor, whatever its scale.

``check`` prints one line per tensor and returns it in ``report``: max-abs,
the worst element's share of its bound, how many elements exceed
2e-2 + u without their allowances (``slack``), the relative Frobenius error
and the worst row's relative error.
"""
import os

import numpy as np
import torch

import paper_2411_06465_amd as L
import workloads as W
from oracle import layer as OL
from oracle.bf16 import from_bits

MAX_ABS = 2e-2
REL_FROB = 5e-3
ROW_REL = 2e-2
TAIL = 6.0          # standard deviations of the contraction allowance


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def host_f64(t):
    if t.dtype == torch.bfloat16:
        return from_bits(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
    return t.detach().double().cpu().numpy()


def bf16_ulp(ref):
    """Spacing of the bf16 grid at |ref| (8 significant bits)."""
    a = np.abs(np.asarray(ref, np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.ldexp(1.0, (np.maximum(e, -126) - 7).astype(np.int64)), 0.0)


def errors(got, ref, bf16=True, allow=None, abs_bound=None, contraction=True):
    """Statistics of got against ref under the bar above: dict with max_abs,
    worst (largest |got - ref| / element bound, or 0 without one), slack
    (elements above the bound without A and C), n (elements), rel_frob,
    row_rel (worst row's error over its floored norm) and ok."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = np.abs(got - ref)
    out = dict(max_abs=0.0, worst=0.0, slack=0, n=int(d.size), rel_frob=0.0, row_rel=0.0, ok=True)
    if d.size == 0:
        return out
    out["max_abs"] = float(np.max(d))
    base = None
    extra = 0.0 if allow is None else np.asarray(allow, np.float64)
    if bf16:
        base = MAX_ABS + bf16_ulp(np.maximum(np.abs(got), np.abs(ref)))
        if contraction and ref.ndim >= 1:
            extra = extra + contraction_allowance(ref)
    elif abs_bound is not None:
        base = np.full(ref.shape, float(abs_bound))
    ok = True
    if base is not None:
        bound = base + extra
        out["worst"] = float(np.max(d / bound))
        out["slack"] = int(np.count_nonzero(d > base))
        ok &= bool(np.all(d <= bound))
    den = float(np.linalg.norm(ref))
    num = float(np.linalg.norm(got - ref))
    out["rel_frob"] = num / den if den > 0 else num
    ok &= out["rel_frob"] <= REL_FROB
    if ref.ndim >= 2 and ref.shape[-1] > 1:
        r2 = ref.reshape(-1, ref.shape[-1])
        e2 = (got - ref).reshape(-1, ref.shape[-1])
        rn = np.linalg.norm(r2, axis=1)
        floor = den / np.sqrt(r2.shape[0])
        out["row_rel"] = float(np.max(np.linalg.norm(e2, axis=1) / np.maximum(rn, floor))) if floor > 0 else 0.0
        ok &= out["row_rel"] <= ROW_REL
    out["ok"] = bool(ok)
    return out


def check(name, got, ref, bf16=True, allow=None, abs_bound=None, contraction=True, report=None):
    """The parity bar above; prints and records one line per tensor."""
    e = errors(got, ref, bf16, allow, abs_bound, contraction)
    line = (f"{name:>14s}: max_abs {e['max_abs']:.3e}  worst {e['worst']:.3f}  slack {e['slack']:>6d}/{e['n']:<10d} "
            f"rel_frob {e['rel_frob']:.3e}  row_rel {e['row_rel']:.3e}  {'ok' if e['ok'] else 'FAIL'}")
    if report is not None:
        report.append(line)
    print(line, flush=True)
    return e["ok"]


def keep_report(title, lines):
    """Append a case's lines to the file named by L4D_PARITY_REPORT (if set)."""
    path = os.environ.get("L4D_PARITY_REPORT")
    if not path:
        return
    with open(path, "a") as f:
        f.write(title + "\n")
        for ln in lines:
            f.write("  " + ln + "\n")


# ------------------------------------------------------------------ the layer

def _rstd(x, eps):
    return 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def contraction_allowance(ref):
    """C of a contraction output: TAIL x REL_FROB x the RMS of each row."""
    return TAIL * REL_FROB * np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))


def layer_allowances(w, wbits, fw, bw):
    """Per-element allowance A of the outputs that take a stored bf16 operand
    elementwise.  An operand o that is itself a contraction output may deviate
    by its own bound u(o) + C(o); one that is not (x, the input) only by a flip
    u(o).  A is the first-order image of those deviations:
      xn2  = g2 h1 rstd2      : |g2| rstd2 (u(h1) + C(h1))
      act  = silu(G)          : |silu'(G)| (u(G) + C(G))
      prod = silu(G) U        : |silu'(G) U| (u(G) + C(G)) + |silu(G)| (u(U) + C(U))
      y    = h1 + f           : u(h1)           (f and the rest of h1: C of y's row)
    dx has none: its terms dh1 (residual copy), d(xn2) and d(xn1) are kept in
    fp32, and the bf16 gradients reach it only through products (C of dx's
    row).  Rows are own SP rows, except act and prod over the local tokens."""
    u, C = bf16_ulp, contraction_allowance
    g1, g2 = from_bits(wbits["norm1"]), from_bits(wbits["norm2"])
    r1, r2 = _rstd(fw["x"], w.rms_eps), _rstd(fw["h1"], w.rms_eps)
    G, U = fw["gate"], fw["up"]
    sg = 1.0 / (1.0 + np.exp(-G))
    dsilu = sg * (1.0 + G * (1.0 - sg))
    eg, eu = u(G) + C(G), u(U) + C(U)
    a = dict(xn2=np.abs(g2) * r2 * (u(fw["h1"]) + C(fw["h1"])),
             act=np.abs(dsilu) * eg,
             prod=np.abs(dsilu * U) * eg + np.abs(G * sg) * eu,
             y=u(fw["h1"]))
    return a


# stash tensors computed elementwise from stored operands (no contraction allowance)
ELEMENTWISE = ("xn1", "xn2", "act", "prod")


def compare_layer(w, buf, saved, fw, bw):
    """Every stashed tensor, output, weight gradient, remote dK/dV and send of
    one layer call against the oracle.  Returns (ok, report lines)."""
    al = layer_allowances(w, buf.wbits, fw, bw)
    rep, ok = [], True
    same_x = np.array_equal(host_f64(saved["x"]), fw["x"])
    rep.append(f"{'stash.x':>14s}: {'bit-exact copy of the input' if same_x else 'DIFFERS from the input'}")
    print(rep[-1], flush=True)
    ok &= same_x
    for n in ("xn1", "q", "k", "v", "ctx", "h1", "xn2", "gate", "up", "act", "prod"):
        ok &= check("stash." + n, host_f64(saved[n]), fw[n], allow=al.get(n), contraction=n not in ELEMENTWISE,
                    report=rep)
    ok &= check("lse", host_f64(saved["lse"]), fw["lse"], bf16=False, abs_bound=MAX_ABS, report=rep)
    ok &= check("y", host_f64(buf.y), fw["y"], allow=al["y"], report=rep)
    ok &= check("dx", host_f64(buf.dx), bw["dx"], report=rep)
    for n in ("norm1", "qkv", "o", "norm2", "gate_up", "down"):
        ok &= check("d_" + n, host_f64(buf.grads[n]), bw["d_" + n], bf16=False, report=rep)
    if w.cp > 1:
        ok &= check("d_remote_k", host_f64(buf.d_remote[0]), bw["d_remote_k"], report=rep)
        ok &= check("d_remote_v", host_f64(buf.d_remote[1]), bw["d_remote_v"], report=rep)
    if w.tp > 1:
        ok &= check("o_send", host_f64(saved["o_partial"]), fw["o_send"], report=rep)
        ok &= check("ffn_send", host_f64(saved["ffn_partial"]), fw["ffn_send"], report=rep)
        ok &= check("dxn2_send", host_f64(buf.sends["dxn2_partial"]), bw["dxn2_send"], report=rep)
        ok &= check("dxn1_send", host_f64(buf.sends["dxn1_partial"]), bw["dxn1_send"], report=rep)
    return ok, rep


class Buffers:
    """Device copies of one workload's inputs plus output buffers."""

    def __init__(self, w: W.LayerWorkload, seed_suffix=""):
        self.w = w
        self.wbits = W.layer_weights(w)
        self.abits = W.layer_activations(w)
        self.weights = {k: dev_bf16(v) for k, v in self.wbits.items()}
        self.x = dev_bf16(self.abits["x"])
        self.dy = dev_bf16(self.abits["dy"])
        self.peers = {k: dev_bf16(v) for k, v in self.abits["peers"].items()}
        b, h = w.micro_batch, w.hidden
        self.y = torch.empty((b, w.s_sp, h), dtype=torch.bfloat16, device="cuda")
        self.dx = torch.empty_like(self.y)
        self.grads = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in self.wbits.items()}
        self.d_remote = None
        if w.cp > 1:
            shape = (b, w.seq - w.s_c, w.k_t * w.d_h)
            self.d_remote = (torch.empty(shape, dtype=torch.bfloat16, device="cuda"),
                             torch.empty(shape, dtype=torch.bfloat16, device="cuda"))
        self.sends = None
        if w.tp > 1:
            shape = (b, (w.tp - 1) * w.s_sp, h)
            self.sends = {n: torch.empty(shape, dtype=torch.bfloat16, device="cuda") for n in L.PEER_OUTPUTS}
        self.model = L.make_model(**w.model())
        self.par = L.make_parallel(**w.parallel())
        f, bw = L.l4d_layer_workspace_bytes(self.model, self.par)
        m = L.mem_estimate(self.model, self.par)
        need = 2 * m["act_bytes_per_layer"] + 4 * w.micro_batch * w.a_t * w.s_c + f + bw + (64 << 20)
        self.arena_buf = torch.empty(need, dtype=torch.uint8, device="cuda")
        self.arena = L.Arena.on(self.arena_buf)

    def stash_view(self, stash, name, shape, dtype=torch.bfloat16):
        ptr, nbytes = stash.tensor(name)
        off = ptr - self.arena_buf.data_ptr()
        return self.arena_buf[off:off + nbytes].view(dtype).view(shape)

    def run(self, keep_stash=True):
        w = self.w
        st = L.llama_layer_fwd(self.model, self.par, self.weights, self.x, self.y, self.arena,
                               peers=self.peers, sends=self.sends)
        saved = {}
        if keep_stash:
            b, d = w.micro_batch, w.d_h
            shapes = dict(x=(b, w.s_sp, w.hidden), xn1=(b, w.s_sp, w.hidden), h1=(b, w.s_sp, w.hidden),
                          xn2=(b, w.s_sp, w.hidden), q=(b, w.s_c, w.a_t * d), ctx=(b, w.s_c, w.a_t * d),
                          k=(b, w.s_c, w.k_t * d), v=(b, w.s_c, w.k_t * d), gate=(b, w.s_c, w.f_t),
                          up=(b, w.s_c, w.f_t), act=(b, w.s_c, w.f_t), prod=(b, w.s_c, w.f_t))
            for n, shp in shapes.items():
                saved[n] = self.stash_view(st, n, shp).clone()
            saved["lse"] = self.stash_view(st, "lse", (b, w.a_t, w.s_c), torch.float32).clone()
            saved["_bytes"] = st.bytes()
            fwd_sends = {n: self.sends[n].clone() for n in ("o_partial", "ffn_partial")} if self.sends else {}
        L.llama_layer_bwd(self.model, self.par, self.weights, st, self.dy, self.dx, self.grads, self.arena,
                          peers=self.peers, sends=self.sends,
                          d_remote_k=self.d_remote[0] if self.d_remote else None,
                          d_remote_v=self.d_remote[1] if self.d_remote else None)
        torch.cuda.synchronize()
        if keep_stash:
            saved.update(fwd_sends)
        return saved


def oracle_layer(w: W.LayerWorkload, wbits, abits):
    sh = OL.Shard(**w.shard_kwargs())
    wts = {k: from_bits(v) for k, v in wbits.items()}
    peers = {k: from_bits(v) for k, v in abits["peers"].items()}
    x, dy = from_bits(abits["x"]), from_bits(abits["dy"])
    fw = OL.layer_forward(sh, wts, x, peers)
    bw = OL.layer_backward(sh, wts, fw, dy, peers)
    return fw, bw
