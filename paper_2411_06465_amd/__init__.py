"""Thin Python binding of libl4d.so (the C ABI in include/l4d.h).

Argument marshalling only: every step of the layer runs in the HIP library.
Tensors are torch tensors on the GPU (device memory and streams are the only
things torch provides here); the functions keep the C names.  The library is
loaded from this directory; if it is missing, every call raises.
"""
import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# L4D_LIB names another build of the same sources (the host-sanitizer build of the tests)
LIB_PATH = os.environ.get("L4D_LIB") or os.path.join(_HERE, "libl4d.so")

L4D_OK, L4D_EINVAL, L4D_ENOMEM, L4D_EDEVICE = 0, 1, 2, 3
STASH_NAMES = ["x", "xn1", "q", "k", "v", "ctx", "h1", "xn2", "gate", "up", "act", "prod", "lse"]
HEAD_STASH_NAMES = ["x", "xn", "probs"]
EMB_STASH_NAMES = ["ids"]


class L4DError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"l4d error {code}: {msg}")
        self.code = code


class Model(C.Structure):
    _fields_ = [("hidden", C.c_int64), ("n_heads", C.c_int64), ("n_kv_heads", C.c_int64),
                ("ffn", C.c_int64), ("n_layers", C.c_int64), ("vocab", C.c_int64),
                ("rms_eps", C.c_float), ("rope_base", C.c_float)]


class Parallel(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("seq", "micro_batch", "tp", "cp", "pp", "dp", "tp_rank", "cp_rank")]


class Mem(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in ("params_per_gpu", "weight_bytes", "grad_bytes", "optim_bytes",
                                          "act_bytes_per_layer", "act_bytes", "total_bytes")] + \
               [("inexact", C.c_uint32)]


class LayerWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("norm1", "qkv", "o", "norm2", "gate_up", "down")]


class LayerGrads(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("norm1", "qkv", "o", "norm2", "gate_up", "down")]


PEER_INPUTS = ("remote_k", "remote_v", "sp_peer_xn1", "sp_peer_xn2", "sp_peer_o", "sp_peer_ffn",
               "sp_peer_dy", "sp_peer_dh1", "sp_peer_dxn2", "sp_peer_dxn1", "cp_peer_dk", "cp_peer_dv")
PEER_OUTPUTS = ("o_partial", "ffn_partial", "dxn2_partial", "dxn1_partial")


class PeerInputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in PEER_INPUTS]


class PeerOutputs(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in PEER_OUTPUTS]


class Adam(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float), ("grad_scale", C.c_float), ("grad_scale_dev", C.c_void_p),
                ("step", C.c_int64), ("zero_grad", C.c_int32)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        P, i64, u64, f32 = C.c_void_p, C.c_int64, C.c_uint64, C.c_float
        sig = {
            "l4d_last_error": ([], C.c_char_p),
            "mem_estimate": ([C.POINTER(Model), C.POINTER(Parallel), C.POINTER(Mem)], C.c_int),
            "mem_fit": ([C.POINTER(Mem), u64, C.POINTER(C.c_int)], C.c_int),
            "l4d_arena_create": ([P, u64, C.POINTER(P)], C.c_int),
            "l4d_arena_destroy": ([P], C.c_int),
            "l4d_arena_stats": ([P, C.POINTER(u64), C.POINTER(u64), C.POINTER(u64)], C.c_int),
            "l4d_stash_reserve": ([P, C.POINTER(Model), C.POINTER(Parallel), C.POINTER(P)], C.c_int),
            "l4d_stash_bytes": ([P, C.POINTER(u64), C.POINTER(u64), C.POINTER(u64)], C.c_int),
            "l4d_stash_tensor": ([P, C.c_int, C.POINTER(P), C.POINTER(u64)], C.c_int),
            "l4d_stash_release": ([P, P], C.c_int),
            "l4d_layer_workspace_bytes": ([C.POINTER(Model), C.POINTER(Parallel), C.POINTER(u64), C.POINTER(u64)], C.c_int),
            "l4d_lm_head_workspace_bytes": ([i64, i64, i64, C.POINTER(u64)], C.c_int),
            "llama_layer_fwd": ([C.POINTER(Model), C.POINTER(Parallel), C.POINTER(LayerWeights), P,
                                 C.POINTER(PeerInputs), C.POINTER(PeerOutputs), P, P, C.POINTER(P), P], C.c_int),
            "llama_layer_bwd": ([C.POINTER(Model), C.POINTER(Parallel), C.POINTER(LayerWeights),
                                 C.POINTER(PeerInputs), C.POINTER(PeerOutputs), P, P, P, C.POINTER(LayerGrads),
                                 P, P, P, P], C.c_int),
            "lm_head_xent": ([i64, i64, i64, i64, P, P, P, P, P, f32, P, P, P, P, P], C.c_int),
            "lm_head_xent_noalloc": ([i64, i64, i64, i64, P, P, P, P, P, f32, P, P, P, P], C.c_int),
            "l4d_adam_step": ([C.POINTER(Adam), i64, P, P, P, P, P, P], C.c_int),
            "embedding_fwd": ([C.POINTER(Model), C.POINTER(Parallel), P, P, P, P, P, P, C.POINTER(P), P], C.c_int),
            "embedding_bwd": ([C.POINTER(Model), C.POINTER(Parallel), P, P, P, P, P, P], C.c_int),
            "lm_head_fwd": ([C.POINTER(Model), C.POINTER(Parallel), P, P, P, P, P, P, P, P, P, C.POINTER(P), P],
                            C.c_int),
            "lm_head_bwd": ([C.POINTER(Model), C.POINTER(Parallel), P, P, P, P, P, P, f32, P, P, P, P, P, P],
                            C.c_int),
            "l4d_profile_enable": ([C.c_int], C.c_int),
            "l4d_profile_only": ([C.c_char_p], C.c_int),
            "l4d_profile_read": ([C.c_char_p, C.POINTER(i64), C.POINTER(C.c_double)], C.c_int),
            "l4d_profile_dump": ([C.c_char_p, u64, C.POINTER(u64)], C.c_int),
            "l4d_profile_order": ([C.c_char_p, u64, C.POINTER(u64)], C.c_int),
            "l4d_profile_reset": ([], C.c_int),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes, fn.restype = args, res
        _lib = L
    return _lib


def _check(rc):
    if rc != L4D_OK:
        raise L4DError(rc, lib().l4d_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def make_model(hidden, n_heads, n_kv_heads, ffn, n_layers=1, vocab=8, rms_eps=1e-5, rope_base=1e4, **_):
    return Model(hidden, n_heads, n_kv_heads, ffn, n_layers, vocab, rms_eps, rope_base)


def make_parallel(seq, micro_batch=1, tp=1, cp=1, pp=1, dp=1, tp_rank=0, cp_rank=0, **_):
    return Parallel(seq, micro_batch, tp, cp, pp, dp, tp_rank, cp_rank)


# ------------------------------------------------------------------ memory estimate

def mem_estimate(model, par):
    out = Mem()
    _check(lib().mem_estimate(C.byref(model), C.byref(par), C.byref(out)))
    return {n: getattr(out, n) for n, _ in Mem._fields_}


FIT_CLASSES = {0: "fits", 1: "near_limit", 2: "oom"}


def mem_fit(est, device_bytes):
    """'fits' (estimate <= 80% of device_bytes), 'near_limit' (<= 100%) or 'oom';
    `est` is a dict from mem_estimate."""
    m = Mem(*[est[n] for n, _ in Mem._fields_])
    out = C.c_int()
    _check(lib().mem_fit(C.byref(m), device_bytes, C.byref(out)))
    return FIT_CLASSES[out.value]


# ------------------------------------------------------------------ arena / stash

class Arena:
    """Host bookkeeping over caller-owned device memory [base, base + capacity)."""

    def __init__(self, base_ptr, capacity):
        self.h = C.c_void_p()
        _check(lib().l4d_arena_create(C.c_void_p(base_ptr), capacity, C.byref(self.h)))

    @classmethod
    def on(cls, buf):
        """Arena over a torch uint8 device tensor (kept alive by the arena)."""
        a = cls(buf.data_ptr(), buf.numel() * buf.element_size())
        a.buf = buf
        return a

    def stats(self):
        u, p, c = C.c_uint64(), C.c_uint64(), C.c_uint64()
        _check(lib().l4d_arena_stats(self.h, C.byref(u), C.byref(p), C.byref(c)))
        return dict(in_use=u.value, peak=p.value, capacity=c.value)

    def destroy(self):
        if self.h:
            _check(lib().l4d_arena_destroy(self.h))
            self.h = C.c_void_p()


class Stash:
    def __init__(self, handle, arena, names=STASH_NAMES):
        self.h, self.arena, self.names = handle, arena, names

    def bytes(self):
        f, a, p = C.c_uint64(), C.c_uint64(), C.c_uint64()
        _check(lib().l4d_stash_bytes(self.h, C.byref(f), C.byref(a), C.byref(p)))
        return dict(formula=f.value, aux=a.value, padding=p.value)

    def tensor(self, which):
        """(device address, bytes) of stashed tensor `which` (index or name)."""
        if isinstance(which, str):
            which = self.names.index(which)
        ptr, n = C.c_void_p(), C.c_uint64()
        _check(lib().l4d_stash_tensor(self.h, which, C.byref(ptr), C.byref(n)))
        return ptr.value, n.value

    def release(self):
        if self.h:
            _check(lib().l4d_stash_release(self.arena.h, self.h))
            self.h = None


def l4d_stash_reserve(arena, model, par):
    h = C.c_void_p()
    _check(lib().l4d_stash_reserve(arena.h, C.byref(model), C.byref(par), C.byref(h)))
    return Stash(h, arena)


def l4d_layer_workspace_bytes(model, par):
    f, b = C.c_uint64(), C.c_uint64()
    _check(lib().l4d_layer_workspace_bytes(C.byref(model), C.byref(par), C.byref(f), C.byref(b)))
    return f.value, b.value


def l4d_lm_head_workspace_bytes(n, h, v_t):
    b = C.c_uint64()
    _check(lib().l4d_lm_head_workspace_bytes(n, h, v_t, C.byref(b)))
    return b.value


# ------------------------------------------------------------------ layer

def _weights(w):
    return LayerWeights(*[w[n].data_ptr() for n in ("norm1", "qkv", "o", "norm2", "gate_up", "down")])


def _peers(peers):
    peers = peers or {}
    return PeerInputs(*[(peers[n].data_ptr() if peers.get(n) is not None else None) for n in PEER_INPUTS])


def _sends(sends):
    sends = sends or {}
    return PeerOutputs(*[(sends[n].data_ptr() if sends.get(n) is not None else None) for n in PEER_OUTPUTS])


def llama_layer_fwd(model, par, weights, x, y, arena, peers=None, sends=None, stream=None):
    """Forward of one layer shard; returns the Stash for the backward."""
    st = C.c_void_p()
    pi, so = _peers(peers), _sends(sends)
    _check(lib().llama_layer_fwd(C.byref(model), C.byref(par), C.byref(_weights(weights)), _ptr(x),
                                 C.byref(pi), C.byref(so), _ptr(y), arena.h, C.byref(st), _stream(stream)))
    return Stash(st, arena)


def llama_layer_bwd(model, par, weights, stash, dy, dx, grads, arena, peers=None, sends=None,
                    d_remote_k=None, d_remote_v=None, stream=None):
    g = LayerGrads(*[grads[n].data_ptr() for n in ("norm1", "qkv", "o", "norm2", "gate_up", "down")])
    pi, so = _peers(peers), _sends(sends)
    _check(lib().llama_layer_bwd(C.byref(model), C.byref(par), C.byref(_weights(weights)), C.byref(pi),
                                 C.byref(so), stash.h, _ptr(dy), _ptr(dx), C.byref(g), _ptr(d_remote_k),
                                 _ptr(d_remote_v), arena.h, _stream(stream)))
    stash.h = None


def lm_head_xent(hidden, w_lm, targets, loss, d_hidden, d_w_lm, arena, vocab_start=0, peer_lse=None,
                 peer_target_logit=None, grad_scale=1.0, stream=None):
    n, h = hidden.shape
    v_t = w_lm.shape[0]
    _check(lib().lm_head_xent(n, h, v_t, vocab_start, _ptr(hidden), _ptr(w_lm), _ptr(targets), _ptr(peer_lse),
                              _ptr(peer_target_logit), grad_scale, _ptr(loss), _ptr(d_hidden), _ptr(d_w_lm),
                              arena.h, _stream(stream)))


def lm_head_xent_noalloc(hidden, w_lm, targets, loss, d_hidden, d_w_lm, vocab_start=0, peer_lse=None,
                         peer_target_logit=None, grad_scale=1.0, stream=None):
    """lm_head_xent with the library's per-GPU static workspace instead of an arena."""
    n, h = hidden.shape
    v_t = w_lm.shape[0]
    _check(lib().lm_head_xent_noalloc(n, h, v_t, vocab_start, _ptr(hidden), _ptr(w_lm), _ptr(targets),
                                      _ptr(peer_lse), _ptr(peer_target_logit), grad_scale, _ptr(loss),
                                      _ptr(d_hidden), _ptr(d_w_lm), _stream(stream)))


# ------------------------------------------------------------------ the ends of the model

def embedding_fwd(model, par, ids, w_emb, x_out, arena, receipt=None, send=None, stream=None):
    """Vocabulary-parallel lookup of the rank's b*s_c tokens; returns the Stash (the ids)."""
    st = C.c_void_p()
    _check(lib().embedding_fwd(C.byref(model), C.byref(par), _ptr(ids), _ptr(w_emb), _ptr(receipt), _ptr(send),
                               _ptr(x_out), arena.h, C.byref(st), _stream(stream)))
    return Stash(st, arena, EMB_STASH_NAMES)


def embedding_bwd(model, par, stash, dx, d_w_emb, arena, peer_dx=None, stream=None):
    _check(lib().embedding_bwd(C.byref(model), C.byref(par), stash.h, _ptr(dx), _ptr(peer_dx), _ptr(d_w_emb),
                               arena.h, _stream(stream)))
    stash.h = None


def lm_head_fwd(model, par, x, w_norm, w_lm, targets, loss, arena, peer_xn=None, peer_lse=None,
                peer_target_logit=None, stream=None):
    """Final RMSNorm, logits (FP32) and cross-entropy; returns the Stash (x, xn, softmax)."""
    st = C.c_void_p()
    _check(lib().lm_head_fwd(C.byref(model), C.byref(par), _ptr(x), _ptr(w_norm), _ptr(w_lm), _ptr(targets),
                             _ptr(peer_xn), _ptr(peer_lse), _ptr(peer_target_logit), _ptr(loss), arena.h,
                             C.byref(st), _stream(stream)))
    return Stash(st, arena, HEAD_STASH_NAMES)


def lm_head_bwd(model, par, w_norm, w_lm, targets, stash, dx, d_w_norm, d_w_lm, arena, grad_scale=1.0,
                peer_xn=None, peer_dxn=None, dxn_send=None, stream=None):
    _check(lib().lm_head_bwd(C.byref(model), C.byref(par), _ptr(w_norm), _ptr(w_lm), _ptr(targets), _ptr(peer_xn),
                             _ptr(peer_dxn), _ptr(dxn_send), grad_scale, stash.h, _ptr(dx), _ptr(d_w_norm),
                             _ptr(d_w_lm), arena.h, _stream(stream)))
    stash.h = None


# ------------------------------------------------------------------ optimizer step

def l4d_adam_step(grad, master, m, v, weight, step, lr, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0,
                  grad_scale=1.0, grad_scale_dev=None, zero_grad=False, n=None, stream=None):
    """One Adam step over a shard: grad, master, m, v fp32 and weight bf16, all of
    n elements (default: grad.numel()), updated in place."""
    n = grad.numel() if n is None else n
    hp = Adam(lr, beta1, beta2, eps, weight_decay, grad_scale,
              None if grad_scale_dev is None else grad_scale_dev.data_ptr(), step, 1 if zero_grad else 0)
    _check(lib().l4d_adam_step(C.byref(hp), n, _ptr(grad), _ptr(master), _ptr(m), _ptr(v), _ptr(weight),
                               _stream(stream)))


# ------------------------------------------------------------------ kernel timing

def l4d_profile_enable(on=True):
    _check(lib().l4d_profile_enable(1 if on else 0))


def l4d_profile_only(name=None):
    _check(lib().l4d_profile_only(name.encode() if name else None))


def l4d_profile_reset():
    _check(lib().l4d_profile_reset())


def l4d_profile_read(name=None):
    n, ms = C.c_int64(), C.c_double()
    _check(lib().l4d_profile_read(name.encode() if name else None, C.byref(n), C.byref(ms)))
    return n.value, ms.value


def l4d_profile_dump():
    need = C.c_uint64()
    _check(lib().l4d_profile_dump(None, 0, C.byref(need)))
    buf = C.create_string_buffer(need.value + 1)
    _check(lib().l4d_profile_dump(buf, need.value + 1, C.byref(need)))
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out


def l4d_profile_order():
    """Labels of the timed launches since the last reset, in launch order."""
    need = C.c_uint64()
    _check(lib().l4d_profile_order(None, 0, C.byref(need)))
    buf = C.create_string_buffer(need.value + 1)
    _check(lib().l4d_profile_order(buf, need.value + 1, C.byref(need)))
    return buf.value.decode().split()
