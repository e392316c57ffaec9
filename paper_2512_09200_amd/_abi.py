"""ctypes mirror of include/lattice.h and the loader of liblattice.so.

Argument marshalling only: every computation runs in the HIP library.  The
library must have been built (``python -m paper_2512_09200_amd.build``);
loading fails loudly otherwise.
"""
import ctypes
import os
from ctypes import POINTER, Structure, c_char_p, c_float, c_int, c_int32, c_int64, c_size_t, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblattice.so")

MAX_LAYERS = 8
NOALLOC_SCRATCH_BYTES = 256 << 20
F32, BF16 = 0, 1
POOL_SUM, POOL_MEAN = 0, 1
DOT, FM, STACK = 0, 1, 2
FP8_ROWWISE, FP8_TENSORWISE = 0, 1
ACT_RELU, ACT_SWISHRN, ACT_HARDSWISHRN = 0, 1, 2
BLOCKNORM_COLS = 128

STATUS = {0: "OK", 1: "INVALID_ARG", 2: "UNSUPPORTED", 3: "WORKSPACE", 4: "BAD_INPUT", 5: "HIP"}


class lattice_jagged(Structure):
    _fields_ = [("num_features", c_int32), ("batch", c_int32), ("offsets", c_void_p),
                ("indices", c_void_p), ("nnz", c_int64)]


class lattice_tables(Structure):
    _fields_ = [("data", c_void_p), ("dtype", c_int), ("dim", c_int32), ("total_rows", c_int64),
                ("row_base", c_void_p), ("max_rows", c_int64)]


class lattice_sparse_grad(Structure):
    _fields_ = [("unique_rows", c_void_p), ("seg_offsets", c_void_p), ("sorted_bags", c_void_p),
                ("num_unique", c_void_p), ("grad_rows", c_void_p)]


class lattice_stack_layer(Structure):
    _fields_ = [("W", c_void_p), ("A", c_void_p), ("C", c_void_p), ("gamma", c_void_p),
                ("dW", c_void_p), ("dA", c_void_p), ("dC", c_void_p), ("dgamma", c_void_p),
                ("L", c_void_p), ("dL", c_void_p)]


class lattice_interact_desc(Structure):
    _fields_ = [("kind", c_int), ("dtype", c_int), ("n", c_int32), ("dim", c_int32),
                ("rank", c_int32), ("emit_slot0", c_int32), ("fm_W", c_void_p),
                ("fm_dW", c_void_p), ("n_layers", c_int32), ("stack_n", c_int32),
                ("ln_eps", c_float), ("layers", POINTER(lattice_stack_layer)), ("lcb_n", c_int32),
                ("slot_mask", c_void_p), ("fp8_proj", c_int32), ("skip_absent", c_int32)]


class lattice_stack_state(Structure):
    _fields_ = [(k, c_int64 * MAX_LAYERS) for k in ("P", "F", "H", "mean", "rstd", "Xn")]


class lattice_linear(Structure):
    _fields_ = [("in_dim", c_int32), ("out_dim", c_int32), ("W", c_void_p), ("b", c_void_p),
                ("dW", c_void_p), ("db", c_void_p), ("gain", c_void_p), ("dgain", c_void_p),
                ("pre", c_void_p), ("rinv", c_void_p)]


class lattice_mlp_desc(Structure):
    _fields_ = [("dtype", c_int), ("n_layers", c_int32), ("layers", POINTER(lattice_linear)),
                ("relu_last", c_int32), ("act", c_int), ("norm_block", c_int32), ("norm_eps", c_float),
                ("tower_heads", c_int32), ("n_domains", c_int32), ("untied_layers", c_int32),
                ("domain_offsets", POINTER(c_int64))]


class lattice_loss_desc(Structure):
    _fields_ = [("labels", c_void_p), ("mask", c_void_p), ("loss", c_void_p),
                ("d_logits", c_void_p), ("d_logits_op", c_void_p)]


class lattice_model_desc(Structure):
    _fields_ = [("dtype", c_int), ("pool", c_int), ("tables", lattice_tables),
                ("num_features", c_int32), ("dense_in", c_int32), ("bottom", lattice_mlp_desc),
                ("interact", lattice_interact_desc), ("top", lattice_mlp_desc)]


class lattice_batch_desc(Structure):
    _fields_ = [("bags", lattice_jagged), ("dense", c_void_p), ("labels", c_void_p),
                ("mask", c_void_p), ("domain_offsets", POINTER(c_int64))]


SIDE_EVENTS = 6


class lattice_step_opts(Structure):
    _fields_ = [("lr_tables", c_float), ("emit_grad_rows", c_int32), ("nnz_capacity", c_int64),
                ("stage_events", POINTER(c_void_p)), ("side_stream", c_void_p),
                ("side_events", POINTER(c_void_p)), ("fp8_top", c_int32)]


STAGES = ["embbag_fwd", "bottom_fwd", "interact_fwd", "top_fwd", "loss", "top_bwd",
          "interact_bwd", "top_wgrad", "bottom_bwd", "embbag_sort", "embbag_runs", "embbag_reduce",
          "embbag_fixup"]


class lattice_step_layout(Structure):
    _fields_ = ([("total_bytes", c_int64), ("X", c_int64), ("t", c_int64), ("t_stride", c_int64),
                 ("logits", c_int64), ("d_logits", c_int64), ("d_logits_op", c_int64),
                 ("loss", c_int64), ("d_t", c_int64), ("dX", c_int64),
                 ("bottom_act", c_int64 * MAX_LAYERS), ("top_act", c_int64 * MAX_LAYERS),
                 ("top_grad", c_int64 * MAX_LAYERS), ("bottom_grad", c_int64 * MAX_LAYERS),
                 ("top_pre", c_int64 * MAX_LAYERS), ("top_rinv", c_int64 * MAX_LAYERS),
                 ("top_gout", c_int64 * MAX_LAYERS)]
                + [(k, c_int64) for k in ("unique_rows", "seg_offsets", "sorted_bags",
                                          "num_unique", "grad_rows", "interact", "scratch",
                                          "scratch_bytes", "sparse", "sparse_bytes", "fp8",
                                          "fp8_bytes")])


# (name, restype, argtypes)
_SIGS = [
    ("lattice_embbag_fwd", c_int, [POINTER(lattice_tables), POINTER(lattice_jagged), c_int, c_void_p,
                                   c_int, c_int32, c_int32, c_void_p]),
    ("lattice_embbag_bwd_workspace", c_size_t, [POINTER(lattice_tables), POINTER(lattice_jagged)]),
    ("lattice_embbag_bwd", c_int, [POINTER(lattice_tables), POINTER(lattice_jagged), c_int, c_void_p,
                                   c_int, c_int32, c_int32, POINTER(lattice_sparse_grad), c_float,
                                   c_void_p, c_size_t, c_void_p]),
    ("lattice_embbag_bwd_noalloc", c_int, [POINTER(lattice_tables), POINTER(lattice_jagged), c_int,
                                           c_void_p, c_int, c_int32, c_int32,
                                           POINTER(lattice_sparse_grad), c_float, c_void_p]),
    ("lattice_validate_batch", c_int, [POINTER(lattice_tables), POINTER(lattice_jagged),
                                       POINTER(c_int64), c_void_p]),
    ("lattice_interact_workspace", c_size_t, [POINTER(lattice_interact_desc), c_int32]),
    ("lattice_interact_fwd", c_int, [POINTER(lattice_interact_desc), c_int32, c_void_p, c_void_p,
                                     c_int64, c_void_p, c_size_t, c_void_p]),
    ("lattice_interact_bwd", c_int, [POINTER(lattice_interact_desc), c_int32, c_void_p, c_void_p,
                                     c_int64, c_void_p, c_void_p, c_size_t, c_void_p]),
    ("lattice_mlp_heads_workspace", c_size_t, [POINTER(lattice_mlp_desc), c_int32]),
    ("lattice_mlp_heads_fwd", c_int, [POINTER(lattice_mlp_desc), c_int32, c_void_p, c_int64,
                                      POINTER(c_void_p), POINTER(c_int64), POINTER(lattice_loss_desc),
                                      c_void_p, c_size_t, c_void_p]),
    ("lattice_mlp_heads_bwd", c_int, [POINTER(lattice_mlp_desc), c_int32, c_void_p, c_int64,
                                      POINTER(c_void_p), POINTER(c_int64), c_void_p, c_int64,
                                      c_void_p, c_int64, c_void_p, c_size_t, c_void_p]),
    ("lattice_fp8_quantize_workspace", c_size_t, []),
    ("lattice_fp8_quantize", c_int, [c_void_p, c_int, c_int64, c_int64, c_int64, c_int, c_void_p, c_int64,
                                     c_void_p, c_void_p, c_size_t, c_void_p]),
    ("lattice_linear_fp8_fwd", c_int, [c_void_p, c_int64, c_void_p, c_int, c_void_p, c_int64, c_void_p, c_int,
                                       c_void_p, c_int32, c_int32, c_int32, c_int32, c_int32, c_void_p,
                                       c_int, c_int64, c_void_p]),
    ("lattice_step_plan", c_int, [POINTER(lattice_model_desc), c_int32, c_int64,
                                  POINTER(lattice_step_opts), POINTER(lattice_step_layout)]),
    ("lattice_interact_state", c_int, [POINTER(lattice_interact_desc), c_int32, POINTER(lattice_stack_state)]),
    ("lattice_step", c_int, [POINTER(lattice_model_desc), POINTER(lattice_batch_desc),
                             POINTER(lattice_step_opts), c_void_p, c_size_t, c_void_p]),
    ("lattice_forward", c_int, [POINTER(lattice_model_desc), POINTER(lattice_batch_desc),
                                POINTER(lattice_step_opts), c_void_p, c_size_t, c_void_p]),
    ("lattice_status_string", c_char_p, [c_int]),
    ("lattice_last_error", c_char_p, []),
    ("lattice_abi_version", c_int, []),
]
EXPORTED = [s[0] for s in _SIGS]

_lib = None


class LatticeError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def load():
    """Load liblattice.so (built in-tree); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2512_09200_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, res, args in _SIGS:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def check(status):
    if status != 0:
        msg = load().lattice_last_error().decode(errors="replace")
        raise LatticeError(status, msg)
