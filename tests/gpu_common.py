"""Helpers shared by the GPU parity tests: upload the seeded inputs, run the
library through its C ABI, run the oracle on the same bytes, and compare."""
import numpy as np
import torch

import paper_2411_06465_amd as L
import workloads as W
from oracle import layer as OL
from oracle.bf16 import from_bits

# Parity bar for floating point outputs (bf16 storage, fp32 accumulation).
#   fp32 outputs: relative Frobenius error <= 5e-3.
#   bf16 outputs: relative Frobenius error <= 5e-3, and
#     * at least 99% of the elements within 2e-2 plus one bf16 step of the
#       reference (the output's own rounding), and
#     * every element within 2e-2 plus four bf16 steps at the tensor's largest
#       magnitude.
# The second clause is for rounding at a boundary: a stored bf16 operand rounds
# one step away from the oracle's where its fp32 sum lands next to a rounding
# boundary (about one element in a thousand at full size), and the step moves
# every value computed from it -- by one operand-sized step, which for a sum
# with cancellation (y = h1 + f, dx = dh1 + ...) is many steps of the result.
# A wrong index, tile or mask moves a block of elements by their own size and
# fails the Frobenius bound or the cap.
MAX_ABS = 2e-2
REL_FROB = 5e-3
TIGHT_FRACTION = 0.99
CAP_STEPS = 4


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


def errors(got, ref):
    """(max |got - ref|, fraction of elements within 2e-2 + one bf16 step of ref,
    max |got - ref| minus the cap 2e-2 + CAP_STEPS steps at max |ref|,
    relative Frobenius error)."""
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = np.abs(got - ref)
    if d.size == 0:
        return 0.0, 1.0, 0.0, 0.0
    max_abs = float(np.max(d))
    tight = float(np.mean(d <= MAX_ABS + bf16_ulp(ref)))
    cap = MAX_ABS + CAP_STEPS * float(bf16_ulp(np.max(np.abs(ref))))
    den = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(got - ref) / den) if den > 0 else float(np.linalg.norm(got - ref))
    return max_abs, tight, max_abs - cap, rel


def check(name, got, ref, bf16=True, report=None):
    """The parity bar above; prints and records one line per tensor."""
    ma, tight, over_cap, rf = errors(got, ref)
    ok = rf <= REL_FROB and (tight >= TIGHT_FRACTION and over_cap <= 0 if bf16 else True)
    line = (f"{name:>14s}: max_abs {ma:.3e}  within_1step {tight:.5f}  over_cap {over_cap:+.3e}  "
            f"rel_frob {rf:.3e}  {'ok' if ok else 'FAIL'}")
    if report is not None:
        report.append(line)
    print(line, flush=True)
    return ok


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
