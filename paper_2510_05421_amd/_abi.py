"""ctypes declarations for libdvi.so (include/dvi.h).  Argument marshalling only."""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdvi.so")

OK, ERR_ARG, ERR_STATE, ERR_CAPACITY, ERR_DEVICE, ERR_NUMERIC = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "DVI_OK", -1: "DVI_ERR_ARG", -2: "DVI_ERR_STATE", -3: "DVI_ERR_CAPACITY",
                -4: "DVI_ERR_DEVICE", -5: "DVI_ERR_NUMERIC"}
FP32, BF16 = 0, 1
PROBES = {"off": 0, "qkv": 1, "attn_out": 2, "gate_up": 3, "down": 4, "head": 5, "attention": 6}

c_i32, c_f32, c_vp = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p
P_i32 = ctypes.POINTER(ctypes.c_int32)


class Config(ctypes.Structure):
    _fields_ = [("n_layers", c_i32), ("split_k", c_i32), ("d_model", c_i32), ("n_heads", c_i32),
                ("n_kv_heads", c_i32), ("head_dim", c_i32), ("ffn_dim", c_i32), ("vocab", c_i32),
                ("rms_eps", c_f32), ("rope_theta", c_f32), ("max_batch", c_i32), ("max_seq", c_i32),
                ("max_k_spec", c_i32), ("lora_rank", c_i32), ("lora_gamma", c_f32),
                ("buffer_rows", c_i32), ("dtype", c_i32)]


class Weights(ctypes.Structure):
    _fields_ = [("tok_emb", c_vp), ("attn_norm", ctypes.POINTER(c_vp)), ("wq", ctypes.POINTER(c_vp)),
                ("wk", ctypes.POINTER(c_vp)), ("wv", ctypes.POINTER(c_vp)), ("wo", ctypes.POINTER(c_vp)),
                ("mlp_norm", ctypes.POINTER(c_vp)), ("w_gate", ctypes.POINTER(c_vp)),
                ("w_up", ctypes.POINTER(c_vp)), ("w_down", ctypes.POINTER(c_vp)),
                ("final_norm", c_vp), ("lm_head", c_vp), ("lora_A", c_vp), ("lora_B", c_vp)]


class UpdateArgs(ctypes.Structure):
    _fields_ = [("c_kl", c_f32), ("c_ce", c_f32), ("c_pg", c_f32), ("c_ent", c_f32),
                ("tau", c_f32), ("baseline", c_f32), ("lr", c_f32), ("beta1", c_f32), ("beta2", c_f32),
                ("eps", c_f32), ("opt_step", c_i32), ("grad_A_out", c_vp), ("grad_B_out", c_vp)]


class UpdateStats(ctypes.Structure):
    _fields_ = [("loss", c_f32), ("kl", c_f32), ("ce", c_f32), ("pg", c_f32), ("entropy", c_f32),
                ("rows", c_i32), ("accepted", c_i32), ("fresh", c_i32), ("fresh_accepted", c_i32)]


# name -> (restype, argtypes)
SIGNATURES = {
    "dvi_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(Config)]),
    "dvi_create": (c_i32, [ctypes.POINTER(Config), ctypes.POINTER(Weights), c_vp, ctypes.c_size_t, c_vp,
                           ctypes.POINTER(c_vp)]),
    "dvi_destroy": (None, [c_vp]),
    "dvi_prefill": (c_i32, [c_vp, c_i32, c_vp, c_vp, c_i32, c_vp]),
    "dvi_draft": (c_i32, [c_vp, c_i32, c_vp, c_vp]),
    "dvi_verify": (c_i32, [c_vp, c_vp, c_vp]),
    "dvi_verify_static": (c_i32, [c_vp, c_vp, c_vp]),
    "dvi_commit": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]),
    "dvi_decode_steps": (c_i32, [c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp]),
    "dvi_abort_step": (c_i32, [c_vp]),
    "dvi_update_drafter": (c_i32, [c_vp, ctypes.POINTER(UpdateArgs), ctypes.POINTER(UpdateStats)]),
    "dvi_last_error": (ctypes.c_char_p, [c_vp]),
    "dvi_read_kv": (c_i32, [c_vp, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp]),
    "dvi_read_logits": (c_i32, [c_vp, c_vp]),
    "dvi_read_draft_logits": (c_i32, [c_vp, c_vp]),
    "dvi_read_lengths": (c_i32, [c_vp, c_vp]),
    "dvi_buffer_info": (c_i32, [c_vp, c_vp, c_vp]),
    "dvi_read_buffer": (c_i32, [c_vp, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]),
    "dvi_write_buffer": (c_i32, [c_vp, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp]),
    "dvi_get_timings": (c_i32, [c_vp, c_vp, c_vp, c_vp, c_vp]),
    "dvi_set_graphs": (c_i32, [c_vp, c_i32]),
    "dvi_set_sampling": (c_i32, [c_vp, c_f32, ctypes.c_uint64]),
    "dvi_probe_kernel": (c_i32, [c_vp, c_i32]),
    "dvi_probe_read": (c_i32, [c_vp, c_vp, c_vp, c_vp]),
    "dvi_measure_read_rate": (c_i32, [c_vp, c_vp, ctypes.c_size_t, c_i32, c_vp]),
}

_lib = None


def load():
    """Load libdvi.so; raises if the HIP library was not built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libdvi.so is not built (%s); run __graft_entry__.build() or "
                              "python paper_2510_05421_amd/build.py" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


class DVIError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), msg))
        self.status = status
