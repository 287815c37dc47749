"""ctypes binding of libhpd.so: the C ABI of include/hpd.h, names unchanged.

Argument marshalling only: every step of the decode path runs in the HIP
kernels of the library.  Device pointers are plain integers (for torch
tensors, ``tensor.data_ptr()``); streams are hipStream_t handles as integers
(``torch.cuda.current_stream().cuda_stream``) or None for the null stream.
There is no fallback: if the library is missing, loading fails loudly.
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhpd.so")

HPD_MAX_K = 16
HPD_HEAD_DIM = 64
HPD_NOALLOC_SCRATCH_BYTES = 32 << 20   # static scratch of hpd_branch_attn_step_noalloc
HPD_F32, HPD_BF16 = 0, 1
STATUS = {0: "HPD_OK", 1: "HPD_ERR_INVALID_ARGUMENT", 2: "HPD_ERR_UNSUPPORTED",
          3: "HPD_ERR_WORKSPACE_TOO_SMALL", 4: "HPD_ERR_HIP", 5: "HPD_ERR_HOST_ALLOC",
          6: "HPD_ERR_OUT_OF_BLOCKS"}

# Work-item record widths and fields (paper_2607_18839_amd/csrc/plan.h).
SI_NFIELDS = PI_NFIELDS = 12
SI = dict(page=0, kvh=1, row0=2, nrows=3, key0=4, key1=5, slot=6, flags=7, prefix_row=8,
          page_q_row=9, page_rows=10, pos=11)
PI = dict(branch=0, kvh=1, row0=2, nrows=3, key0=4, key1=5, slot=6, past=7, priv_row=8,
          q_row=9, num_new=10)

c_i32p = ctypes.POINTER(ctypes.c_int32)
c_i64p = ctypes.POINTER(ctypes.c_int64)


class HpdError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class hpd_attn_desc(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


class hpd_paged_kv(ctypes.Structure):
    _fields_ = [("block_rows", ctypes.c_int32), ("num_blocks", ctypes.c_int32), ("num_entries", ctypes.c_int32),
                ("blocks", c_i32p), ("page_block0", c_i32p), ("branch_block0", c_i32p)]


class hpd_batch_desc(ctypes.Structure):
    _fields_ = [("num_pages", ctypes.c_int32), ("prefix_len", c_i32p), ("prefix_row", c_i64p),
                ("num_branches", ctypes.c_int32), ("branch_page", c_i32p), ("num_new", c_i32p),
                ("past_len", c_i32p), ("priv_row", c_i64p), ("fork_len", c_i32p),
                ("paged", ctypes.POINTER(hpd_paged_kv))]


class hpd_plan_info(ctypes.Structure):
    _fields_ = [("num_tokens", ctypes.c_int32), ("num_pages", ctypes.c_int32),
                ("num_branches", ctypes.c_int32), ("q_row", c_i32p), ("priv_row", c_i64p),
                ("prefix_row", c_i64p), ("page_q_row", c_i32p), ("page_T", c_i32p),
                ("visible", c_i32p), ("shared_rows", ctypes.c_int64), ("priv_rows", ctypes.c_int64),
                ("num_shared_items", ctypes.c_int32), ("num_private_items", ctypes.c_int32),
                ("shared_items", c_i32p), ("private_items", c_i32p), ("token_slots", c_i32p),
                ("num_partial_slots", ctypes.c_int64), ("pos_token", c_i32p)]


PP = ctypes.POINTER(ctypes.c_void_p)


class hpd_model_desc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("intermediate", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("w_qkv", PP), ("w_o", PP), ("w_gate", PP), ("w_up", PP), ("w_down", PP),
                ("g_attn_norm", PP), ("g_mlp_norm", PP), ("weight_format", ctypes.c_int32),
                ("q_norm", PP), ("k_norm", PP), ("rope_theta", ctypes.c_float)]


HPD_WEIGHTS_TORCH, HPD_WEIGHTS_PACKED = 0, 1


class hpd_pmtp_desc(ctypes.Structure):
    _fields_ = [("vocab", ctypes.c_int32), ("draft_inner", ctypes.c_int32), ("lm_head", ctypes.c_void_p),
                ("g_final", ctypes.c_void_p), ("embed", ctypes.c_void_p), ("w_draft_gate_up", ctypes.c_void_p),
                ("w_draft_down", ctypes.c_void_p), ("window", ctypes.c_int32)]


class hpd_sched_config(ctypes.Structure):
    _fields_ = [("num_blocks", ctypes.c_int32), ("block_rows", ctypes.c_int32), ("kv_threshold", ctypes.c_double),
                ("window", ctypes.c_int32), ("max_active", ctypes.c_int32), ("fork_token", ctypes.c_int32),
                ("child_token", ctypes.c_int32), ("eos_token", ctypes.c_int32)]


class hpd_sched_batch(ctypes.Structure):
    _fields_ = [("num_pages", ctypes.c_int32), ("num_branches", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("prefix_len", c_i32p), ("branch_page", c_i32p), ("num_new", c_i32p), ("past_len", c_i32p),
                ("fork_len", c_i32p), ("paged", hpd_paged_kv), ("request", c_i32p), ("tokens_in", c_i32p),
                ("prefill_from", c_i32p), ("prefill_to", c_i32p), ("num_preempted", ctypes.c_int32),
                ("preempted", c_i32p), ("num_admitted", ctypes.c_int32), ("admitted", c_i32p)]


# Every symbol include/hpd.h declares, with its ctypes signature.
SIGNATURES = {
    "hpd_plan_create": (ctypes.c_int, [ctypes.POINTER(hpd_attn_desc), ctypes.POINTER(hpd_batch_desc),
                                       ctypes.POINTER(ctypes.c_void_p)]),
    "hpd_plan_destroy": (None, [ctypes.c_void_p]),
    "hpd_plan_workspace_bytes": (ctypes.c_size_t, [ctypes.c_void_p]),
    "hpd_plan_query": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(hpd_plan_info)]),
    "hpd_plan_upload": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "hpd_branch_attn_step": (ctypes.c_int, [ctypes.c_void_p] + [ctypes.c_void_p] * 6 +
                             [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "hpd_decode_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(hpd_model_desc), ctypes.c_void_p]),
    "hpd_decode_step": (ctypes.c_int, [ctypes.POINTER(hpd_model_desc), ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, PP, PP, PP, PP, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_void_p]),
    "hpd_packed_weight_bytes": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32]),
    "hpd_pack_weight": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p]),
    "hpd_pack_weight_f16": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p]),
    "hpd_pack_gate_up": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_void_p, ctypes.c_void_p]),
    "hpd_branch_attn_step_noalloc": (ctypes.c_int, [ctypes.c_void_p] * 8 + [ctypes.c_void_p]),
    "hpd_kernel_timing": (ctypes.c_int, [ctypes.c_int, ctypes.c_int]),
    "hpd_attn_phase_isolation": (ctypes.c_int, [ctypes.c_int]),
    "hpd_pmtp_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(hpd_model_desc), ctypes.POINTER(hpd_pmtp_desc),
                                                   ctypes.c_void_p]),
    "hpd_verify_draft_step": (ctypes.c_int, [ctypes.POINTER(hpd_model_desc), ctypes.POINTER(hpd_pmtp_desc),
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                             ctypes.c_void_p]),
    "hpd_embed_tokens": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "hpd_kv_pool_create": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p)]),
    "hpd_kv_pool_destroy": (None, [ctypes.c_void_p]),
    "hpd_kv_pool_free_blocks": (ctypes.c_int32, [ctypes.c_void_p]),
    "hpd_kv_seq_new": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, c_i32p]),
    "hpd_kv_seq_reserve": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]),
    "hpd_kv_seq_truncate": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]),
    "hpd_kv_seq_release": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "hpd_kv_seq_info": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, c_i32p, c_i32p, c_i32p]),
    "hpd_kv_seq_blocks": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, ctypes.c_int32]),
    "hpd_kv_batch_tables": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, ctypes.c_int32, c_i32p,
                                           c_i32p, ctypes.c_int32, c_i32p, c_i32p, c_i32p]),
    "hpd_sched_create": (ctypes.c_int, [ctypes.POINTER(hpd_sched_config), ctypes.POINTER(ctypes.c_void_p)]),
    "hpd_sched_destroy": (None, [ctypes.c_void_p]),
    "hpd_sched_submit": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, c_i32p]),
    "hpd_sched_schedule": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(hpd_sched_batch)]),
    "hpd_sched_commit": (ctypes.c_int, [ctypes.c_void_p, c_i32p, c_i32p, c_i32p]),
    "hpd_sched_next_output": (ctypes.c_int, [ctypes.c_void_p, c_i32p, c_i32p, ctypes.c_int32, c_i32p]),
    "hpd_sched_counts": (ctypes.c_int, [ctypes.c_void_p, c_i32p, c_i32p, c_i32p]),
    "hpd_sched_request": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, c_i32p, c_i32p, c_i32p, c_i32p]),
    "hpd_kernel_times_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int]),
    "hpd_kernel_kind_name": (ctypes.c_char_p, [ctypes.c_int]),
    "hpd_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "hpd_last_error_message": (ctypes.c_char_p, []),
}

_lib = None


def load(path=LIB_PATH):
    """Load libhpd.so once; raise if it is missing (there is no CPU fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise ImportError(f"{path} not built: run `python -m paper_2607_18839_amd.build` "
                              "(the HIP library is required; there is no fallback path)")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status, what):
    if status != 0:
        msg = load().hpd_last_error_message().decode(errors="replace")
        raise HpdError(status, msg if msg.startswith(what) else f"{what}: {msg}")


def _i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def _i64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int64)


def _ptr(a, ty):
    return None if a is None else a.ctypes.data_as(ty)


class Plan:
    """Owns an hpd_plan handle (host memory), built by hpd_plan_create."""

    def __init__(self, handle, attn):
        self.handle = handle
        self.attn = attn

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.hpd_plan_destroy(self.handle)
            self.handle = None

    @property
    def workspace_bytes(self):
        return int(load().hpd_plan_workspace_bytes(self.handle))


def hpd_plan_create(num_q_heads, num_kv_heads, prefix_len, branch_page, num_new, past_len,
                    head_dim=HPD_HEAD_DIM, softmax_scale=0.0, dtype=HPD_BF16, out_dtype=None,
                    prefix_row=None, priv_row=None, fork_len=None, paged=None):
    """paged: None, or a dict with block_rows, num_blocks, blocks, page_block0,
    branch_block0 (hpd_paged_kv)."""
    lib = load()
    attn = hpd_attn_desc(num_q_heads, num_kv_heads, head_dim, softmax_scale, dtype,
                         dtype if out_dtype is None else out_dtype)
    arrs = dict(prefix_len=_i32(prefix_len), branch_page=_i32(branch_page), num_new=_i32(num_new),
                past_len=_i32(past_len), prefix_row=_i64(prefix_row), priv_row=_i64(priv_row),
                fork_len=_i32(fork_len))
    pg = None
    if paged is not None:
        for k in ("blocks", "page_block0", "branch_block0"):
            arrs["pg_" + k] = _i32(paged[k])
        pg = hpd_paged_kv(int(paged["block_rows"]), int(paged["num_blocks"]), len(arrs["pg_blocks"]),
                          _ptr(arrs["pg_blocks"], c_i32p), _ptr(arrs["pg_page_block0"], c_i32p),
                          _ptr(arrs["pg_branch_block0"], c_i32p))
    batch = hpd_batch_desc(len(arrs["prefix_len"]), _ptr(arrs["prefix_len"], c_i32p),
                           _ptr(arrs["prefix_row"], c_i64p), len(arrs["num_new"]),
                           _ptr(arrs["branch_page"], c_i32p), _ptr(arrs["num_new"], c_i32p),
                           _ptr(arrs["past_len"], c_i32p), _ptr(arrs["priv_row"], c_i64p),
                           _ptr(arrs["fork_len"], c_i32p), None if pg is None else ctypes.pointer(pg))
    h = ctypes.c_void_p()
    _check(lib.hpd_plan_create(ctypes.byref(attn), ctypes.byref(batch), ctypes.byref(h)), "hpd_plan_create")
    return Plan(h, attn)


def hpd_plan_query(plan):
    """The plan's integer bookkeeping and work lists as numpy arrays (copies)."""
    info = hpd_plan_info()
    _check(load().hpd_plan_query(plan.handle, ctypes.byref(info)), "hpd_plan_query")
    T, npg, nb = info.num_tokens, info.num_pages, info.num_branches

    def arr(p, n, w=1):
        if n * w == 0:
            return np.zeros((n, w) if w > 1 else n, dtype=np.int64 if p._type_ is ctypes.c_int64 else np.int32)
        a = np.ctypeslib.as_array(p, shape=(n * w,)).copy()
        return a.reshape(n, w) if w > 1 else a

    return dict(T=T, q_row=arr(info.q_row, nb), priv_row=arr(info.priv_row, nb),
                prefix_row=arr(info.prefix_row, npg), page_q_row=arr(info.page_q_row, npg),
                page_T=arr(info.page_T, npg), visible=arr(info.visible, T),
                shared_rows=info.shared_rows, priv_rows=info.priv_rows,
                shared_items=arr(info.shared_items, info.num_shared_items, SI_NFIELDS),
                private_items=arr(info.private_items, info.num_private_items, PI_NFIELDS),
                token_slots=arr(info.token_slots, T, 2), num_partial_slots=info.num_partial_slots,
                pos_token=arr(info.pos_token, T, 2))


def hpd_plan_upload(plan, workspace, nbytes, stream=None):
    _check(load().hpd_plan_upload(plan.handle, workspace, nbytes, stream), "hpd_plan_upload")


def hpd_branch_attn_step(plan, q, shared_k, shared_v, priv_k, priv_v, out, lse, workspace,
                         workspace_bytes, stream=None):
    _check(load().hpd_branch_attn_step(plan.handle, q, shared_k, shared_v, priv_k, priv_v, out, lse,
                                       workspace, workspace_bytes, stream), "hpd_branch_attn_step")


def hpd_branch_attn_step_noalloc(plan, q, shared_k, shared_v, priv_k, priv_v, out, lse, stream=None):
    _check(load().hpd_branch_attn_step_noalloc(plan.handle, q, shared_k, shared_v, priv_k, priv_v, out, lse,
                                               stream), "hpd_branch_attn_step_noalloc")


def _ptr_array(ptrs):
    if ptrs is None:
        return None
    return (ctypes.c_void_p * len(ptrs))(*ptrs)


def model_desc(num_layers, hidden, intermediate, rms_eps, w_qkv, w_o, w_gate, w_up, w_down,
               g_attn_norm=None, g_mlp_norm=None, weight_format=HPD_WEIGHTS_TORCH, q_norm=None, k_norm=None,
               rope_theta=0.0):
    """hpd_model_desc from lists of device pointers; keeps the arrays alive."""
    keep = [_ptr_array(x) for x in (w_qkv, w_o, w_gate, w_up, w_down, g_attn_norm, g_mlp_norm, q_norm, k_norm)]
    cast = [None if k is None else ctypes.cast(k, PP) for k in keep]
    d = hpd_model_desc(num_layers, hidden, intermediate, rms_eps, *cast[:7], weight_format, *cast[7:],
                       float(rope_theta))
    d._keep = keep
    return d


def hpd_packed_weight_bytes(rows, cols):
    return int(load().hpd_packed_weight_bytes(rows, cols))


def hpd_pack_weight(w, rows, cols, out, stream=None):
    _check(load().hpd_pack_weight(w, rows, cols, out, stream), "hpd_pack_weight")


def hpd_pack_weight_f16(w, rows, cols, out, stream=None):
    _check(load().hpd_pack_weight_f16(w, rows, cols, out, stream), "hpd_pack_weight_f16")


def hpd_pack_gate_up(w_gate, w_up, intermediate, hidden, out, stream=None):
    _check(load().hpd_pack_gate_up(w_gate, w_up, intermediate, hidden, out, stream), "hpd_pack_gate_up")


def hpd_decode_workspace_bytes(model, plan):
    return int(load().hpd_decode_workspace_bytes(ctypes.byref(model), plan.handle))


def hpd_decode_step(model, plan, hidden_in, hidden_out, shared_k, shared_v, priv_k, priv_v,
                    workspace, workspace_bytes, stream=None):
    arrs = [_ptr_array(x) for x in (shared_k, shared_v, priv_k, priv_v)]
    _check(load().hpd_decode_step(ctypes.byref(model), plan.handle, hidden_in, hidden_out,
                                  *[ctypes.cast(a, PP) for a in arrs], workspace, workspace_bytes,
                                  stream), "hpd_decode_step")


HPD_NUM_KERNEL_KINDS = 14


class hpd_kernel_times(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int64 * HPD_NUM_KERNEL_KINDS),
                ("total_ms", ctypes.c_double * HPD_NUM_KERNEL_KINDS), ("dropped", ctypes.c_int64)]


def hpd_kernel_timing(enable, max_launches=8192):
    _check(load().hpd_kernel_timing(int(bool(enable)), max_launches), "hpd_kernel_timing")


def hpd_kernel_times_read(keep_pairs=False):
    """{kind name: (launch count, total ms)} since the previous read."""
    t = hpd_kernel_times()
    _check(load().hpd_kernel_times_read(ctypes.byref(t), int(bool(keep_pairs))), "hpd_kernel_times_read")
    lib = load()
    out = {lib.hpd_kernel_kind_name(k).decode(): (int(t.count[k]), float(t.total_ms[k]))
           for k in range(HPD_NUM_KERNEL_KINDS)}
    out["_dropped"] = (int(t.dropped), 0.0)
    return out


def declared_symbols(header=None):
    """Function names declared in include/hpd.h."""
    import re
    header = header or os.path.join(os.path.dirname(_HERE), "include", "hpd.h")
    text = open(header).read()
    return sorted(set(re.findall(r"\b(hpd_[a-z_]+)\s*\(", text)))


def hpd_attn_phase_isolation(enable):
    _check(load().hpd_attn_phase_isolation(1 if enable else 0), "hpd_attn_phase_isolation")


class KvPool:
    """hpd_kv_pool: host manager of paged K/V block ids (the device pools are
    the caller's).  Sequences are roots (a page's prefix) or branches forked
    from a root."""

    def __init__(self, num_blocks, block_rows):
        h = ctypes.c_void_p()
        _check(load().hpd_kv_pool_create(num_blocks, block_rows, ctypes.byref(h)), "hpd_kv_pool_create")
        self.handle, self.num_blocks, self.block_rows = h, int(num_blocks), int(block_rows)

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.hpd_kv_pool_destroy(self.handle)
            self.handle = None

    def free_blocks(self):
        return int(load().hpd_kv_pool_free_blocks(self.handle))

    def new(self, parent=-1, fork_len=0):
        out = ctypes.c_int32()
        _check(load().hpd_kv_seq_new(self.handle, parent, fork_len, ctypes.byref(out)), "hpd_kv_seq_new")
        return out.value

    def reserve(self, seq, new_len):
        _check(load().hpd_kv_seq_reserve(self.handle, seq, new_len), "hpd_kv_seq_reserve")

    def truncate(self, seq, new_len):
        _check(load().hpd_kv_seq_truncate(self.handle, seq, new_len), "hpd_kv_seq_truncate")

    def release(self, seq):
        _check(load().hpd_kv_seq_release(self.handle, seq), "hpd_kv_seq_release")

    def info(self, seq):
        v = [ctypes.c_int32() for _ in range(4)]
        _check(load().hpd_kv_seq_info(self.handle, seq, *[ctypes.byref(x) for x in v]), "hpd_kv_seq_info")
        return dict(len=v[0].value, num_blocks=v[1].value, parent=v[2].value, fork_len=v[3].value)

    def blocks(self, seq):
        n = self.info(seq)["num_blocks"]
        out = np.zeros(max(n, 1), np.int32)
        _check(load().hpd_kv_seq_blocks(self.handle, seq, _ptr(out, c_i32p), n), "hpd_kv_seq_blocks")
        return out[:n]

    def batch_tables(self, page_seqs, branch_seqs):
        """hpd_paged_kv fields (a dict for hpd_plan_create's `paged`)."""
        ps, bs = _i32(page_seqs), _i32(branch_seqs)
        n = ctypes.c_int32()
        p0, b0 = np.zeros(max(len(ps), 1), np.int32), np.zeros(max(len(bs), 1), np.int32)
        lib = load()
        st = lib.hpd_kv_batch_tables(self.handle, len(ps), _ptr(ps, c_i32p), len(bs), _ptr(bs, c_i32p), None, 0,
                                     _ptr(p0, c_i32p), _ptr(b0, c_i32p), ctypes.byref(n))
        blocks = np.zeros(max(n.value, 1), np.int32)
        if st != 0 or n.value > 0:
            _check(lib.hpd_kv_batch_tables(self.handle, len(ps), _ptr(ps, c_i32p), len(bs), _ptr(bs, c_i32p),
                                           _ptr(blocks, c_i32p), n.value, _ptr(p0, c_i32p), _ptr(b0, c_i32p),
                                           ctypes.byref(n)), "hpd_kv_batch_tables")
        return dict(block_rows=self.block_rows, num_blocks=self.num_blocks, blocks=blocks[:n.value],
                    page_block0=p0[:len(ps)], branch_block0=b0[:len(bs)])


class Sched:
    """hpd_sched: the host scheduler of the inference workflow (FCFS with
    hierarchical parallel decoding) and the K/V block pool it owns."""

    def __init__(self, num_blocks, block_rows, kv_threshold, window, max_active, fork_token, child_token,
                 eos_token):
        cfg = hpd_sched_config(num_blocks, block_rows, kv_threshold, window, max_active, fork_token, child_token,
                               eos_token)
        h = ctypes.c_void_p()
        _check(load().hpd_sched_create(ctypes.byref(cfg), ctypes.byref(h)), "hpd_sched_create")
        self.handle, self.window = h, int(window)
        self.num_blocks, self.block_rows = int(num_blocks), int(block_rows)

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.hpd_sched_destroy(self.handle)
            self.handle = None

    def submit(self, prompt_len, first_token, max_new):
        out = ctypes.c_int32()
        _check(load().hpd_sched_submit(self.handle, prompt_len, first_token, max_new, ctypes.byref(out)),
               "hpd_sched_submit")
        return out.value

    def schedule(self):
        """The next step's batch as a dict of numpy copies (hpd_sched_batch)."""
        b = hpd_sched_batch()
        _check(load().hpd_sched_schedule(self.handle, ctypes.byref(b)), "hpd_sched_schedule")

        def arr(p, n):
            return np.ctypeslib.as_array(p, shape=(n,)).copy() if n > 0 else np.zeros(0, np.int32)

        npg, nb, T = b.num_pages, b.num_branches, b.num_tokens
        out = dict(num_pages=npg, num_branches=nb, num_tokens=T, prefix_len=arr(b.prefix_len, npg),
                   branch_page=arr(b.branch_page, nb), num_new=arr(b.num_new, nb), past_len=arr(b.past_len, nb),
                   fork_len=arr(b.fork_len, nb), request=arr(b.request, nb), tokens_in=arr(b.tokens_in, T),
                   prefill_from=arr(b.prefill_from, nb), prefill_to=arr(b.prefill_to, nb),
                   preempted=arr(b.preempted, b.num_preempted), admitted=arr(b.admitted, b.num_admitted))
        out["paged"] = None if nb == 0 else dict(
            block_rows=b.paged.block_rows, num_blocks=b.paged.num_blocks,
            blocks=arr(b.paged.blocks, b.paged.num_entries), page_block0=arr(b.paged.page_block0, npg),
            branch_block0=arr(b.paged.branch_block0, nb))
        return out

    def commit(self, verified, n_acc, draft_out):
        """Host arrays: verified [T], n_acc [nb], draft_out [nb][HPD_MAX_K]."""
        v, n = _i32(verified), _i32(n_acc)
        d = None if draft_out is None else np.ascontiguousarray(draft_out, dtype=np.int32)
        if d is not None and d.size and d.shape[-1] != HPD_MAX_K:
            raise ValueError("draft_out must be [num_branches][HPD_MAX_K]")
        _check(load().hpd_sched_commit(self.handle, _ptr(v, c_i32p) if v is not None and v.size else None,
                                       _ptr(n, c_i32p) if n is not None and n.size else None,
                                       _ptr(d, c_i32p) if d is not None and d.size else None), "hpd_sched_commit")

    def next_output(self):
        """(page id, tokens) of the oldest finished page, or None."""
        lib = load()
        page, n = ctypes.c_int32(), ctypes.c_int32()
        _check(lib.hpd_sched_next_output(self.handle, ctypes.byref(page), None, 0, ctypes.byref(n)),
               "hpd_sched_next_output")
        if page.value < 0:
            return None
        if n.value == 0:   # an empty page was taken by the query itself
            return page.value, np.zeros(0, np.int32)
        buf = np.zeros(n.value, np.int32)
        _check(lib.hpd_sched_next_output(self.handle, ctypes.byref(page), _ptr(buf, c_i32p), n.value,
                                         ctypes.byref(n)), "hpd_sched_next_output")
        return page.value, buf[:n.value]

    def counts(self):
        v = [ctypes.c_int32() for _ in range(3)]
        _check(load().hpd_sched_counts(self.handle, *[ctypes.byref(x) for x in v]), "hpd_sched_counts")
        return dict(waiting=v[0].value, active=v[1].value, free_blocks=v[2].value)

    def request(self, rid):
        v = [ctypes.c_int32() for _ in range(4)]
        _check(load().hpd_sched_request(self.handle, rid, *[ctypes.byref(x) for x in v]), "hpd_sched_request")
        return dict(state=("waiting", "active", "done")[v[0].value], len=v[1].value, kept=v[2].value,
                    recorded=v[3].value)


def hpd_pmtp_workspace_bytes(model, pmtp, plan):
    return int(load().hpd_pmtp_workspace_bytes(ctypes.byref(model), ctypes.byref(pmtp), plan.handle))


def hpd_verify_draft_step(model, pmtp, plan, hidden, tokens_in, verified, n_acc, draft_out, workspace,
                          workspace_bytes, stream=None):
    _check(load().hpd_verify_draft_step(ctypes.byref(model), ctypes.byref(pmtp), plan.handle, hidden, tokens_in,
                                        verified, n_acc, draft_out, workspace, workspace_bytes, stream),
           "hpd_verify_draft_step")


def hpd_embed_tokens(embed, vocab, hidden, tokens, T, out, stream=None):
    _check(load().hpd_embed_tokens(embed, vocab, hidden, tokens, T, out, stream), "hpd_embed_tokens")
