"""The C ABI of libconduit (include/conduit.h) as ctypes declarations, with no
torch dependency: status codes and enums, the structs, every entry point's
signature, and a loader that applies them.  conduit.py builds the torch-facing
binding on top; host-only checks (the sanitizer build's test) use this alone.
"""
import ctypes as C

# status codes
OK, EINVAL, ENOMEM, EEMPTY, EDEVICE, ESTATE = 0, -1, -2, -3, -4, -5
_STATUS_NAMES = {EINVAL: "EINVAL", ENOMEM: "ENOMEM", EEMPTY: "EEMPTY", EDEVICE: "EDEVICE", ESTATE: "ESTATE"}

# dtypes, transforms, columns
U8, I32, F32, BF16 = 0, 1, 2, 3
XF_NONE, XF_U8_F32, XF_U8_BF16_NORM, XF_TOKENS_PAD = 0, 1, 2, 3
(COL_OBS, COL_ACTION, COL_REWARD, COL_DONE, COL_EPISODE, COL_STEP, COL_LENGTH, COL_AUX, COL_LEAVES, COL_TREE,
 COL_MAX_PRIO) = range(11)

class ConduitError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class BufferOpts(C.Structure):
    _fields_ = [("prioritized", C.c_int32), ("alpha_num", C.c_int32), ("alpha_den", C.c_int32),
                ("beta", C.c_double), ("frame_stack", C.c_int32), ("action_bytes", C.c_int32),
                ("ragged", C.c_int32), ("aux_elem_bytes", C.c_int32), ("payload_placement", C.c_int32),
                ("weight_norm", C.c_int32), ("single_stream", C.c_int32)]


class Transitions(C.Structure):
    _fields_ = [("n", C.c_int64), ("obs", C.c_void_p), ("offsets", C.c_void_p), ("src_elems", C.c_int64),
                ("aux", C.c_void_p),
                ("action", C.c_void_p), ("reward", C.c_void_p), ("done", C.c_void_p),
                ("episode_id", C.c_void_p), ("step", C.c_void_p), ("prio", C.c_void_p)]


class Transform(C.Structure):
    _fields_ = [("kind", C.c_int32), ("channels", C.c_int32), ("mean", C.c_float * 4), ("std", C.c_float * 4),
                ("pad_id", C.c_int32)]


class LearnerBatch(C.Structure):
    _fields_ = [("obs", C.c_void_p), ("action", C.c_void_p), ("reward", C.c_void_p), ("done", C.c_void_p),
                ("mask", C.c_void_p), ("aux", C.c_void_p), ("length", C.c_void_p)]


class SchedCosts(C.Structure):
    _fields_ = [("t_rollout", C.c_double), ("t_update", C.c_double), ("t_sync_ing", C.c_double),
                ("t_sync_del", C.c_double), ("n_ing", C.c_int32), ("n_del", C.c_int32),
                ("g_ing", C.POINTER(C.c_double)), ("t_ing", C.POINTER(C.c_double)),
                ("g_del", C.POINTER(C.c_double)), ("t_del", C.POINTER(C.c_double)), ("on_policy", C.c_int32)]


class SchedMode(C.Structure):
    _fields_ = [("overlap_ing", C.c_int32), ("overlap_del", C.c_int32), ("i_ing", C.c_int32), ("i_del", C.c_int32),
                ("g_ing", C.c_double), ("g_del", C.c_double), ("t_ing_path", C.c_double),
                ("t_del_path", C.c_double), ("t_iter", C.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class OffpolicyLoop(C.Structure):
    _fields_ = [("overlap_ing", C.c_int32), ("g_ing", C.c_int32), ("overlap_del", C.c_int32), ("g_del", C.c_int32),
                ("iters", C.c_int64), ("unit", C.c_int64), ("batch", C.c_int64),
                ("rollout_work", C.c_int64), ("update_work", C.c_int64),
                ("rollout", Transitions), ("uniforms", C.c_void_p), ("new_prio", C.c_void_p),
                ("idx_out", C.c_void_p), ("is_w_out", C.c_void_p), ("xf", C.POINTER(Transform)),
                ("out", LearnerBatch)]


class OnpolicyLoop(C.Structure):
    _fields_ = [("overlap_ing", C.c_int32), ("ing_slices", C.c_int32), ("overlap_del", C.c_int32),
                ("minibatches", C.c_int32), ("iters", C.c_int64), ("steps", C.c_int64), ("envs", C.c_int64),
                ("rollout_work", C.c_int64), ("update_work", C.c_int64),
                ("obs", C.c_void_p), ("reward", C.c_void_p), ("value", C.c_void_p), ("done", C.c_void_p),
                ("bootstrap", C.c_void_p), ("gamma", C.c_double), ("lam", C.c_double), ("perm", C.c_void_p),
                ("xf", C.POINTER(Transform)), ("adv", C.c_void_p), ("ret", C.c_void_p), ("out_obs", C.c_void_p),
                ("out_adv", C.c_void_p), ("out_ret", C.c_void_p)]


PLACE_HBM, PLACE_HOST_PINNED, PLACE_HOST_PAGEABLE = 0, 1, 2
WNORM_BATCH, WNORM_BUFFER = 0, 1
PLACEMENT_NAMES = ("hbm", "host_pinned", "host_pageable")


class PlaceProfile(C.Structure):
    _fields_ = [("bw_in", (C.c_double * 3) * 2), ("bw_out", C.c_double * 3), ("mem", C.c_double * 3)]

    def as_dict(self):
        return {"bw_in_cpu_actor": list(self.bw_in[0]), "bw_in_gpu_actor": list(self.bw_in[1]),
                "bw_out": list(self.bw_out), "mem": list(self.mem)}


class BufferInfo(C.Structure):
    _fields_ = [("capacity", C.c_int64), ("row_bytes", C.c_int64), ("head", C.c_int64), ("size", C.c_int64),
                ("total", C.c_int64), ("tree_depth", C.c_int32), ("tree_nodes", C.c_int64 * 8),
                ("arena_bytes", C.c_int64), ("obs_dtype", C.c_int32), ("prioritized", C.c_int32),
                ("frame_stack", C.c_int32), ("action_bytes", C.c_int32), ("ragged", C.c_int32),
                ("aux_elem_bytes", C.c_int32), ("max_len", C.c_int64)]


CKPT_MAGIC = b"CNDTCKPT"
CKPT_MAX_SECTIONS = 10


class CkptSection(C.Structure):
    _fields_ = [("column", C.c_int32), ("reserved", C.c_int32), ("offset", C.c_int64), ("bytes", C.c_int64)]


class CkptHeader(C.Structure):
    _fields_ = [("magic", C.c_char * 8), ("version", C.c_uint32), ("n_sections", C.c_uint32),
                ("image_bytes", C.c_uint64), ("capacity", C.c_int64), ("row_bytes", C.c_int64),
                ("max_len", C.c_int64), ("obs_dtype", C.c_int32), ("prioritized", C.c_int32),
                ("alpha_num", C.c_int32), ("alpha_den", C.c_int32), ("action_bytes", C.c_int32),
                ("ragged", C.c_int32), ("aux_elem_bytes", C.c_int32), ("reserved", C.c_int32),
                ("head", C.c_int64), ("size", C.c_int64), ("total", C.c_uint64),
                ("section", CkptSection * CKPT_MAX_SECTIONS)]


# every symbol include/conduit.h declares, with its ctypes signature
P = C.c_void_p
I64 = C.c_int64
I32_ = C.c_int32
F64 = C.c_double
ST = C.c_int32
SIGNATURES = {
    "conduit_buffer_opts_default": (None, [P]),
    "conduit_buffer_required_bytes": (C.c_size_t, [I64, P, I32_, I32_, P]),
    "conduit_buffer_create": (ST, [I64, P, I32_, I32_, P, P, C.c_size_t, P]),
    "conduit_buffer_destroy": (None, [P]),
    "conduit_ingest": (ST, [P, P, P]),
    "conduit_update_priorities": (ST, [P, P, P, I64, P]),
    "conduit_sample": (ST, [P, I64, P, P, P, P]),
    "conduit_gather_transform": (ST, [P, P, I64, P, P, P]),
    "conduit_sample_gather": (ST, [P, I64, P, P, P, P, P, P]),
    "conduit_sample_gather_nstep": (ST, [P, I64, P, P, P, P, P, I32_, F64, P, P, P, P, P, P]),
    "conduit_sample_pack_gae": (ST, [P, I64, P, P, P, P, P, P, F64, F64, P, P, P]),
    "conduit_gae": (ST, [P, P, P, P, I64, I64, F64, F64, P, P, P]),
    "conduit_gae_noalloc": (ST, [P, P, P, P, I64, I64, F64, F64, P, P, P]),
    "conduit_update_ingest": (ST, [P, P, P, I64, P, P]),
    "conduit_nstep": (ST, [P, P, I64, I32_, F64, P, P, P, P, P, P, P]),
    "conduit_gae_truncated": (ST, [P, P, P, P, P, P, I64, I64, F64, F64, P, P, P]),
    "conduit_gae_plan": (ST, [I64, I64, I32_, P, P]),
    "conduit_gae_packed": (ST, [P, P, P, I64, I64, F64, F64, P, P, P]),
    "conduit_minibatch_gather": (ST, [P, I64, I64, P, I64, P, P, P, P, I32_, P]),
    "conduit_buffer_get_info": (ST, [P, P]),
    "conduit_buffer_stats": (ST, [P, P, P, P]),
    "conduit_buffer_read": (ST, [P, I32_, I32_, I64, I64, P, P]),
    "conduit_buffer_checkpoint_bytes": (ST, [P, P]),
    "conduit_buffer_checkpoint": (ST, [P, P, C.c_uint64, P]),
    "conduit_buffer_restore": (ST, [P, P, C.c_uint64, P]),
    "conduit_sync_check": (ST, [P, P]),
    "conduit_clear_error": (None, [P]),
    "conduit_last_error": (C.c_char_p, []),
    "conduit_version": (C.c_char_p, []),
    "conduit_schedule": (ST, [P, P, P]),
    "conduit_standin": (ST, [I64, P]),
    "conduit_expand_reference": (ST, [P, P, I64, P]),
    "conduit_sync_cost_us": (ST, [P, P, I32_, P, P]),
    "conduit_sched_candidates": (ST, [I32_, I32_, I32_, I32_, P, I32_, P, P, I32_, P]),
    "conduit_run_onpolicy": (ST, [P, P, P, P, P, P, P]),
    "conduit_placement_profile": (ST, [I64, I32_, P]),
    "conduit_place": (ST, [P, I32_, I64, F64, P, I32_, P, P]),
    "conduit_run_offpolicy": (ST, [P, P, P, P, P, P, P]),
}



def load(path):
    """CDLL of the library at `path` with every declared signature applied."""
    L = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L
