"""ctypes binding of libee.so with the same entry-point names as the C ABI.

Argument marshalling only: every step of the decode path runs in the HIP
kernels behind the ABI. PyTorch, when importable with a GPU, supplies the HIP
stream the library enqueues on."""
import ctypes as C
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_HERE, "libee.so")

EE_F32, EE_BF16 = 0, 1
EE_CAL_EXIT_RATE, EE_CAL_MEDIAN, EE_CAL_NUCLEUS = 0, 1, 2
EE_CONF_MAXPROB, EE_CONF_MARGIN, EE_CONF_NEGENTROPY = 0, 1, 2
EE_FILL_EAGER, EE_FILL_LAZY = 0, 1
_ERRNAMES = {-1: "EE_EINVAL", -2: "EE_ESTATE", -3: "EE_ENOMEM", -4: "EE_EHIP",
             -5: "EE_ECAPACITY", -6: "EE_EDEVICE"}


class EEError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_ERRNAMES.get(code, code)}: {msg}")
        self.code = code


class ee_config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("rope_base", C.c_float), ("rms_eps", C.c_float),
                ("wdtype", C.c_int32), ("max_seq", C.c_int32), ("page_size", C.c_int32)]


class ee_tensor(C.Structure):
    _fields_ = [("name", C.c_char_p), ("ptr", C.c_void_p), ("nbytes", C.c_int64),
                ("on_device", C.c_int32)]


_FP = C.POINTER(C.c_float)
_IP = C.POINTER(C.c_int32)


class ee_debug(C.Structure):
    _fields_ = [("h_exit", _FP), ("h_final", _FP), ("logits_readout", _FP), ("logits_full", _FP),
                ("token", C.c_int32), ("exited", C.c_int32), ("would_exit", C.c_int32),
                ("readout_token", C.c_int32), ("full_token", C.c_int32), ("conf", C.c_float),
                ("conf_full", C.c_float), ("nucleus_mass", C.c_float)]


def _load():
    # torch bundles its own HIP runtime and links it by the unversioned name
    # libamdhip64.so. Loading torch first lets libee.so's libamdhip64.so.7
    # dependency resolve to that same loaded runtime (matched by SONAME), so
    # the process holds exactly one HIP runtime whichever module the caller
    # imports first.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(lib_path):
        raise ImportError(f"{lib_path} is not built; run `python -m paper_2609_14144_amd.build`")
    L = C.CDLL(lib_path)
    V = C.c_void_p
    sig = {
        "ee_create": (C.c_int, [C.POINTER(ee_config), V, C.POINTER(V)]),
        "ee_load_weights": (C.c_int, [V, C.POINTER(ee_tensor), C.c_int32]),
        "ee_prefill": (C.c_int, [V, _IP, C.c_int32, _IP]),
        "ee_decode_step": (C.c_int, [V, C.c_float, C.c_int32, _IP, _IP, _FP]),
        "ee_decode_n": (C.c_int, [V, C.c_float, C.c_int32, C.c_int32, _IP, _IP, _FP]),
        "ee_decode_n_ex": (C.c_int, [V, C.c_float, C.c_int32, C.c_int32, _IP, _IP, _IP, _IP, _FP, _IP]),
        "ee_decode_n_noalloc": (C.c_int, [V, C.c_float, C.c_int32, C.c_int32, V, V, V]),
        "ee_decode_step_ex": (C.c_int, [V, C.c_float, C.c_int32, C.c_int32, C.c_int32, C.POINTER(ee_debug)]),
        "ee_calibrate_threshold": (C.c_int, [V, _IP, _IP, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                             C.c_float, _FP]),
        "ee_calibration_record": (C.c_int, [V, C.c_int32, _FP, _FP]),
        "ee_set_readout_bias": (C.c_int, [V, C.c_int32, _FP, C.c_int32]),
        "ee_set_confidence_measure": (C.c_int, [V, C.c_int32]),
        "ee_refresh": (C.c_int, [V, C.c_int32]),
        "ee_set_fill_policy": (C.c_int, [V, C.c_int32]),
        "ee_set_prefill_chunk": (C.c_int, [V, C.c_int32]),
        "ee_head_eval": (C.c_int, [V, C.c_int32, _FP, _IP, _FP, _FP]),
        "ee_read_kv": (C.c_int, [V, C.c_int32, C.c_int32, _FP, _FP]),
        "ee_set_persistent": (C.c_int, [V, C.c_int32]),
        "ee_set_persistent_grid": (C.c_int, [V, C.c_int32]),
        "ee_last_decode_ms": (C.c_int, [V, _FP]),
        "ee_stream_probe": (C.c_int, [V, C.c_int64, C.c_int32, _FP]),
        "ee_set_timeline": (C.c_int, [V, C.c_int32]),
        "ee_read_timeline": (C.c_int, [V, C.POINTER(C.c_uint64), C.c_int32]),
        "ee_position": (C.c_int32, [V]),
        "ee_reset": (C.c_int, [V]),
        "ee_last_error": (C.c_char_p, [V]),
        "ee_destroy": (None, [V]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


lib = _load()


def _ptr(a, ctype):
    return None if a is None else a.ctypes.data_as(C.POINTER(ctype))


def _torch_stream():
    try:
        import torch
    except ImportError:
        return None
    if not torch.cuda.is_available():
        return None
    return torch.cuda.current_stream().cuda_stream


class Engine:
    """One decode context (one sequence) on the current HIP device."""

    def __init__(self, model, max_seq: int, page_size: int = 64, stream=None):
        self.model = model
        wd = getattr(model, "wdtype")
        self.wdtype = EE_BF16 if wd in ("bf16", EE_BF16) else EE_F32
        cfg = ee_config(model.n_layers, model.hidden, model.n_q_heads, model.n_kv_heads,
                        model.head_dim, model.ffn, model.vocab, float(model.rope_base),
                        float(model.rms_eps), self.wdtype, int(max_seq), int(page_size))
        self.V, self.H, self.L = model.vocab, model.hidden, model.n_layers
        self.max_seq = int(max_seq)
        if stream is None:
            stream = _torch_stream()
        self._ctx = C.c_void_p()
        rc = lib.ee_create(C.byref(cfg), stream, C.byref(self._ctx))
        if rc != 0:
            raise EEError(rc, "ee_create: " + lib.ee_last_error(None).decode())

    # -- helpers -------------------------------------------------------------
    def _check(self, rc):
        if rc != 0:
            raise EEError(rc, lib.ee_last_error(self._ctx).decode())

    def close(self):
        if self._ctx:
            lib.ee_destroy(self._ctx)
            self._ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- ABI mirror -------------------------------------------------------------
    def ee_load_weights(self, weights: dict):
        names, arrs = [], []
        for k, a in weights.items():
            a = np.ascontiguousarray(a)
            names.append(k.encode())
            arrs.append(a)
        ts = (ee_tensor * len(arrs))()
        for i, (n, a) in enumerate(zip(names, arrs)):
            ts[i] = ee_tensor(n, a.ctypes.data, a.nbytes, 0)
        self._check(lib.ee_load_weights(self._ctx, ts, len(arrs)))

    def ee_prefill(self, tokens) -> int:
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        out = C.c_int32(-1)
        self._check(lib.ee_prefill(self._ctx, _ptr(t, C.c_int32), t.size, C.byref(out)))
        return out.value

    def ee_decode_step(self, tau: float, exit_layer: int):
        tok, ex, conf = C.c_int32(), C.c_int32(), C.c_float()
        self._check(lib.ee_decode_step(self._ctx, tau, exit_layer, C.byref(tok), C.byref(ex),
                                       C.byref(conf)))
        return tok.value, bool(ex.value), conf.value

    def ee_decode_n(self, tau: float, exit_layer: int, n: int):
        return self.ee_decode_n_ex(tau, exit_layer, n)[:3]

    def ee_decode_n_ex(self, tau: float, exit_layer: int, n: int, force_tokens=None, force_exit=None):
        ft = None if force_tokens is None else np.ascontiguousarray(force_tokens, dtype=np.int32)
        fe = None if force_exit is None else np.ascontiguousarray(force_exit, dtype=np.int32)
        tok = np.empty(n, np.int32)
        ex = np.empty(n, np.int32)
        conf = np.empty(n, np.float32)
        would = np.empty(n, np.int32)
        self._check(lib.ee_decode_n_ex(self._ctx, tau, exit_layer, n, _ptr(ft, C.c_int32),
                                       _ptr(fe, C.c_int32), _ptr(tok, C.c_int32), _ptr(ex, C.c_int32),
                                       _ptr(conf, C.c_float), _ptr(would, C.c_int32)))
        return tok, ex.astype(bool), conf, would.astype(bool)

    def ee_decode_n_noalloc(self, tau: float, exit_layer: int, n: int, d_tokens: int, d_exited: int,
                            d_conf: int):
        """Outputs go to caller-owned device arrays (raw device addresses, for
        instance torch tensors' data_ptr()): n int32 tokens, n int32 exit
        flags, n float32 confidences."""
        self._check(lib.ee_decode_n_noalloc(self._ctx, tau, exit_layer, n, C.c_void_p(d_tokens),
                                            C.c_void_p(d_exited), C.c_void_p(d_conf)))

    def ee_decode_step_ex(self, tau: float, exit_layer: int, input_token: int = -1,
                          force_exit: int = -1, debug: bool = True) -> dict:
        H, V = self.H, self.V
        bufs = {k: np.full(n, np.nan, np.float32) for k, n in
                (("h_exit", H), ("h_final", H), ("logits_readout", V), ("logits_full", V))}
        d = ee_debug()
        if debug:
            for k, a in bufs.items():
                setattr(d, k, _ptr(a, C.c_float))
        self._check(lib.ee_decode_step_ex(self._ctx, tau, exit_layer, input_token, force_exit,
                                          C.byref(d)))
        out = {k: getattr(d, k) for k in ("token", "exited", "would_exit", "readout_token",
                                          "full_token", "conf", "conf_full", "nucleus_mass")}
        out["exited"] = bool(out["exited"])
        out["would_exit"] = bool(out["would_exit"])
        if debug:
            out.update(bufs)
        return out

    def ee_calibrate_threshold(self, prompts, n_gen: int, exit_layer: int,
                               mode: int = EE_CAL_EXIT_RATE, target: float = 0.5) -> float:
        lens = np.array([len(p) for p in prompts], np.int32)
        flat = np.ascontiguousarray(np.concatenate([np.asarray(p, np.int32) for p in prompts]))
        tau = C.c_float()
        self._check(lib.ee_calibrate_threshold(self._ctx, _ptr(flat, C.c_int32), _ptr(lens, C.c_int32),
                                               len(prompts), n_gen, exit_layer, mode, target,
                                               C.byref(tau)))
        return tau.value

    def ee_calibration_record(self, n: int):
        """(confidences, masses) of the latest calibration's n recorded steps."""
        confs = np.empty(n, np.float32)
        masses = np.empty(n, np.float32)
        self._check(lib.ee_calibration_record(self._ctx, int(n), _ptr(confs, C.c_float), _ptr(masses, C.c_float)))
        return confs, masses

    def ee_set_readout_bias(self, exit_layer: int, b):
        b = np.ascontiguousarray(b, dtype=np.float32)
        self._b_keep = b  # the copy is asynchronous: keep the host buffer alive
        self._check(lib.ee_set_readout_bias(self._ctx, exit_layer, _ptr(b, C.c_float), 0))

    def ee_set_fill_policy(self, policy: int):
        self._check(lib.ee_set_fill_policy(self._ctx, policy))

    def ee_set_prefill_chunk(self, positions: int):
        """0: one position per step (decode program); n > 0: batched chunks of n."""
        self._check(lib.ee_set_prefill_chunk(self._ctx, int(positions)))

    def ee_refresh(self, n: int):
        self._check(lib.ee_refresh(self._ctx, n))

    def ee_set_confidence_measure(self, measure: int):
        self._check(lib.ee_set_confidence_measure(self._ctx, measure))

    def ee_head_eval(self, readout_layer: int, x, want_logits: bool = True):
        x = np.ascontiguousarray(x, dtype=np.float32)
        tok, conf = C.c_int32(), C.c_float()
        lg = np.empty(self.V, np.float32) if want_logits else None
        self._check(lib.ee_head_eval(self._ctx, readout_layer, _ptr(x, C.c_float), C.byref(tok),
                                     C.byref(conf), _ptr(lg, C.c_float)))
        return tok.value, conf.value, lg

    def ee_read_kv(self, layer: int, pos: int):
        n = self.model.n_kv_heads * self.model.head_dim
        k = np.empty(n, np.float32)
        v = np.empty(n, np.float32)
        self._check(lib.ee_read_kv(self._ctx, layer, pos, _ptr(k, C.c_float), _ptr(v, C.c_float)))
        return k, v

    def ee_set_persistent(self, wgs_per_cu):
        """0/False: one kernel per operation; True (or a negative value): the
        persistent kernel with as many workgroups per compute unit as can be
        co-resident; n >= 2: n workgroups per compute unit."""
        if wgs_per_cu is True:
            wgs_per_cu = -1
        self._check(lib.ee_set_persistent(self._ctx, int(wgs_per_cu)))

    def ee_set_persistent_grid(self, nwg: int):
        """Persistent kernel with exactly nwg workgroups."""
        self._check(lib.ee_set_persistent_grid(self._ctx, int(nwg)))

    def ee_set_timeline(self, capacity: int):
        self._check(lib.ee_set_timeline(self._ctx, int(capacity)))
        self._tl_cap = int(capacity)

    def ee_read_timeline(self, n: int = None):
        n = self._tl_cap if n is None else n
        out = np.zeros(n, np.uint64)
        self._check(lib.ee_read_timeline(self._ctx, out.ctypes.data_as(C.POINTER(C.c_uint64)), n))
        return out

    def ee_last_decode_ms(self) -> float:
        ms = C.c_float()
        self._check(lib.ee_last_decode_ms(self._ctx, C.byref(ms)))
        return ms.value

    def ee_stream_probe(self, nbytes: int, reps: int = 5) -> float:
        """Streaming-read ceiling of the device in 1e9 B/s (median of reps launches)."""
        gbps = C.c_float()
        self._check(lib.ee_stream_probe(self._ctx, int(nbytes), int(reps), C.byref(gbps)))
        return gbps.value

    def ee_position(self) -> int:
        return lib.ee_position(self._ctx)

    def ee_reset(self):
        self._check(lib.ee_reset(self._ctx))

    def ee_last_error(self) -> str:
        return lib.ee_last_error(self._ctx).decode()
