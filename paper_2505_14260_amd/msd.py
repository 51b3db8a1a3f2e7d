"""ctypes binding of libmsd.so (the C ABI declared in include/msd.h).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of the library.  PyTorch supplies device memory and the stream.
If the library is missing this module raises -- there is no fallback.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmsd.so")
MAX_TREE = 64

MSD_OK, MSD_ERR_INVALID_ARG, MSD_ERR_CAPACITY, MSD_ERR_STATE, MSD_ERR_HIP = 0, -1, -2, -3, -4
TREE_STATIC, TREE_DYNAMIC = 0, 1

c_i32, c_f32, c_vp, c_sz = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t


class ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", c_i32), ("d_model", c_i32), ("n_heads", c_i32),
                ("n_kv_heads", c_i32), ("head_dim", c_i32), ("ffn_dim", c_i32),
                ("vocab", c_i32), ("rope_theta", c_f32), ("norm_eps", c_f32)]


class Limits(ctypes.Structure):
    _fields_ = [("max_batch", c_i32), ("max_seq", c_i32), ("max_tree", c_i32),
                ("max_prompt", c_i32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down",
                                    "attn_norm", "ffn_norm")]


class TargetWeights(ctypes.Structure):
    _fields_ = [("embed", c_vp), ("layers", ctypes.POINTER(LayerWeights)),
                ("final_norm", c_vp), ("lm_head", c_vp)]


class DraftWeights(ctypes.Structure):
    _fields_ = [("fc", c_vp), ("layer", LayerWeights)]


class Buffers(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in ("target_k", "target_v", "draft_k", "draft_v", "workspace",
                                    "packed_weights")]


class TreeSpec(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("n_nodes", c_i32), ("depth", c_i32), ("topk", c_i32),
                ("parent", ctypes.POINTER(c_i32)), ("rank", ctypes.POINTER(c_i32))]


class TraceRec(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("m", c_i32), ("n", c_i32), ("k", c_i32), ("ms", c_f32)]


class Tree(ctypes.Structure):
    _fields_ = [("n_nodes", c_i32), ("token", c_i32 * MAX_TREE), ("parent", c_i32 * MAX_TREE),
                ("depth", c_i32 * MAX_TREE), ("score", c_f32 * MAX_TREE),
                ("anc", ctypes.c_uint64 * MAX_TREE)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2505_14260_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.msd_buffer_sizes.argtypes = [P(ModelDesc), P(Limits), P(c_sz), P(c_sz), P(c_sz), P(c_sz)]
        L.msd_create.argtypes = [P(ModelDesc), P(Limits), P(TargetWeights), P(DraftWeights),
                                 P(Buffers), c_vp, P(c_vp)]
        L.msd_workspace_size.argtypes = [P(ModelDesc), P(Limits), P(c_sz)]
        L.msd_destroy.argtypes = [c_vp]
        L.msd_last_error.argtypes = [c_vp]
        L.msd_last_error.restype = ctypes.c_char_p
        L.msd_prefill.argtypes = [c_vp, ctypes.c_int, ctypes.c_int, P(c_i32), P(ctypes.c_uint8),
                                  c_vp, P(c_i32)]
        L.msd_draft_tree.argtypes = [c_vp, ctypes.c_int, P(c_i32), P(TreeSpec), c_vp]
        L.msd_verify.argtypes = [c_vp, ctypes.c_int, P(c_i32), c_vp, ctypes.c_int, c_vp, c_vp]
        L.msd_verify_noalloc.argtypes = L.msd_verify.argtypes
        L.msd_accept_compact.argtypes = [c_vp, ctypes.c_int, P(c_i32), c_vp, ctypes.c_int, c_vp,
                                         P(c_i32), P(c_i32), c_vp]
        L.msd_accept_sample.argtypes = [c_vp, ctypes.c_int, P(c_i32), c_vp, ctypes.c_int, c_vp,
                                        ctypes.c_float, ctypes.c_uint64, P(c_i32), P(c_i32),
                                        c_vp]
        L.msd_seq_len.argtypes = [c_vp, ctypes.c_int]
        L.msd_set_state.argtypes = [c_vp, ctypes.c_int, ctypes.c_int, c_vp, c_i32]
        L.msd_set_draft_input.argtypes = [c_vp, ctypes.c_int]
        L.msd_use_caller_weights.argtypes = [c_vp, ctypes.c_int]
        L.msd_stream_read.argtypes = [c_vp, c_sz, ctypes.c_int, c_vp, c_vp]
        L.msd_train_accumulate.argtypes = [c_vp, ctypes.c_int, ctypes.c_int, P(c_i32),
                                           P(ctypes.c_uint8), c_vp, P(ctypes.c_double)]
        L.msd_train_apply.argtypes = [c_vp, ctypes.c_double]
        L.msd_train_read.argtypes = [c_vp, ctypes.c_int, c_vp, c_sz]
        L.msd_train_lr.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                   P(ctypes.c_double)]
        L.msd_train_mix.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, P(c_i32), P(c_i32)]
        L.msd_trace_enable.argtypes = [c_vp, ctypes.c_int, ctypes.c_int]
        L.msd_trace_read.argtypes = [c_vp, ctypes.c_int, P(TraceRec)]
        _lib = L
    return _lib


class MSDError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"msd error {code}: {msg}")
        self.code = code


def _check(ctx, rc):
    if rc != MSD_OK:
        msg = lib().msd_last_error(ctx)
        raise MSDError(rc, msg.decode() if msg else "")


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.POINTER(c_i32))


# --- the C entry points, same names -------------------------------------------------

def msd_buffer_sizes(desc: ModelDesc, lim: Limits):
    t, d, w, p = c_sz(), c_sz(), c_sz(), c_sz()
    _check(None, lib().msd_buffer_sizes(ctypes.byref(desc), ctypes.byref(lim), ctypes.byref(t),
                                        ctypes.byref(d), ctypes.byref(w), ctypes.byref(p)))
    return t.value, d.value, w.value, p.value


def msd_create(desc, lim, tw, dw, bufs, stream):
    out = c_vp()
    _check(None, lib().msd_create(ctypes.byref(desc), ctypes.byref(lim), ctypes.byref(tw),
                                  ctypes.byref(dw), ctypes.byref(bufs), stream, ctypes.byref(out)))
    return out.value


def msd_workspace_size(desc: ModelDesc, lim: Limits):
    w = c_sz()
    _check(None, lib().msd_workspace_size(ctypes.byref(desc), ctypes.byref(lim), ctypes.byref(w)))
    return w.value


def msd_destroy(ctx):
    _check(None, lib().msd_destroy(ctx))


def msd_last_error(ctx):
    m = lib().msd_last_error(ctx)
    return m.decode() if m else ""


def msd_prefill(ctx, seq, tokens, is_visual, visual_ptr):
    tok, ptok = _i32(tokens)
    vis = np.ascontiguousarray(is_visual, dtype=np.uint8)
    first = c_i32()
    _check(ctx, lib().msd_prefill(ctx, seq, len(tok), ptok,
                                  vis.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                  visual_ptr, ctypes.byref(first)))
    return first.value


def msd_draft_tree(ctx, seqs, spec: TreeSpec, trees_ptr):
    s, ps = _i32(seqs)
    _check(ctx, lib().msd_draft_tree(ctx, len(s), ps, ctypes.byref(spec), trees_ptr))


def msd_verify(ctx, seqs, trees_ptr, n_nodes, argmax_ptr, logits_ptr=None):
    s, ps = _i32(seqs)
    _check(ctx, lib().msd_verify(ctx, len(s), ps, trees_ptr, n_nodes, argmax_ptr, logits_ptr))


def msd_verify_noalloc(ctx, seqs, trees_ptr, n_nodes, argmax_ptr, logits_ptr=None):
    s, ps = _i32(seqs)
    _check(ctx, lib().msd_verify_noalloc(ctx, len(s), ps, trees_ptr, n_nodes, argmax_ptr,
                                         logits_ptr))


def msd_accept_compact(ctx, seqs, trees_ptr, n_nodes, argmax_ptr, slot_map_ptr=None):
    s, ps = _i32(seqs)
    emitted = np.zeros((len(s), MAX_TREE), dtype=np.int32)
    n_emit = np.zeros(len(s), dtype=np.int32)
    _check(ctx, lib().msd_accept_compact(
        ctx, len(s), ps, trees_ptr, n_nodes, argmax_ptr,
        emitted.ctypes.data_as(ctypes.POINTER(c_i32)),
        n_emit.ctypes.data_as(ctypes.POINTER(c_i32)), slot_map_ptr))
    return [list(emitted[i, :n_emit[i]]) for i in range(len(s))]


def msd_accept_sample(ctx, seqs, trees_ptr, n_nodes, logits_ptr, temperature, seed,
                      slot_map_ptr=None):
    s, ps = _i32(seqs)
    emitted = np.zeros((len(s), MAX_TREE), dtype=np.int32)
    n_emit = np.zeros(len(s), dtype=np.int32)
    _check(ctx, lib().msd_accept_sample(
        ctx, len(s), ps, trees_ptr, n_nodes, logits_ptr, float(temperature), int(seed),
        emitted.ctypes.data_as(ctypes.POINTER(c_i32)),
        n_emit.ctypes.data_as(ctypes.POINTER(c_i32)), slot_map_ptr))
    return [list(emitted[i, :n_emit[i]]) for i in range(len(s))]


def msd_seq_len(ctx, seq):
    return lib().msd_seq_len(ctx, seq)


# draft input of visual prompt rows (msd_set_draft_input)
DRAFT_VISUAL_INPUTS = {"embedding": 0, "feature": 1}


def msd_set_draft_input(ctx, visual_input):
    _check(ctx, lib().msd_set_draft_input(ctx, visual_input))


def msd_use_caller_weights(ctx, enable):
    _check(ctx, lib().msd_use_caller_weights(ctx, 1 if enable else 0))


def msd_train_accumulate(ctx, seq, tokens, is_visual, visual_ptr):
    """Loss sums (total, regression, token) of one training sequence; its
    gradient sums are added to the context's."""
    tok, ptok = _i32(tokens)
    vis = np.ascontiguousarray(is_visual, dtype=np.uint8)
    loss = (ctypes.c_double * 3)()
    _check(ctx, lib().msd_train_accumulate(ctx, seq, len(tok), ptok,
                                           vis.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                           visual_ptr, loss))
    return tuple(loss)


def msd_train_apply(ctx, lr):
    _check(ctx, lib().msd_train_apply(ctx, lr))


def msd_train_read(ctx, what, out_ptr, n_floats):
    _check(ctx, lib().msd_train_read(ctx, what, out_ptr, n_floats))


def msd_train_lr(step, total_steps, lr_max):
    out = ctypes.c_double()
    _check(None, lib().msd_train_lr(step, total_steps, lr_max, ctypes.byref(out)))
    return out.value


def msd_train_mix(epoch, n_epochs, n_per_epoch):
    nt, nv = c_i32(), c_i32()
    _check(None, lib().msd_train_mix(epoch, n_epochs, n_per_epoch, ctypes.byref(nt),
                                     ctypes.byref(nv)))
    return nt.value, nv.value


def train_param_shapes(dims):
    """Shapes of the trained draft parameters in msd_train_read's order."""
    d, F = dims.d_model, dims.ffn_dim
    qd, kd = dims.n_heads * dims.head_dim, dims.n_kv_heads * dims.head_dim
    return [("fc", (d, 2 * d)), ("wq", (qd, d)), ("wk", (kd, d)), ("wv", (kd, d)),
            ("wo", (d, qd)), ("wg", (F, d)), ("wu", (F, d)), ("wd", (d, F)),
            ("attn_norm", (d,)), ("ffn_norm", (d,))]


def msd_set_state(ctx, seq, L, h_ptr, next_token):
    _check(ctx, lib().msd_set_state(ctx, seq, L, h_ptr, next_token))


def msd_stream_read(buf_ptr, nbytes, workgroups, sink_ptr, stream):
    _check(None, lib().msd_stream_read(buf_ptr, nbytes, workgroups, sink_ptr, stream))


def msd_trace_enable(ctx, capacity, kinds=0xF):
    _check(ctx, lib().msd_trace_enable(ctx, capacity, kinds))


def msd_trace_read(ctx, max_recs=4096):
    recs = (TraceRec * max_recs)()
    n = lib().msd_trace_read(ctx, max_recs, recs)
    if n < 0:
        _check(ctx, n)
    return [(r.kind, r.m, r.n, r.k, r.ms) for r in recs[:n]]


# --- convenience wrapper over device memory held in torch tensors --------------------

def make_static_spec(parent, rank):
    """parent/rank for nodes 1..N (root excluded), canonical order."""
    p, pp = _i32(parent)
    r, pr = _i32(rank)
    depth = np.zeros(len(p) + 1, dtype=np.int32)
    for i, q in enumerate(p, start=1):
        depth[i] = depth[q] + 1
    spec = TreeSpec(TREE_STATIC, len(p), int(depth.max()), 0, pp, pr)
    spec._keep = (p, r)
    return spec


def make_dynamic_spec(topk, depth, n_nodes):
    return TreeSpec(TREE_DYNAMIC, n_nodes, depth, topk, None, None)


class Engine:
    """Owns device copies of the weights and the caller-side buffers."""

    def __init__(self, dims, target, draft, max_batch=1, max_seq=1024, max_tree=64,
                 max_prompt=1024, device="cuda", visual_input="embedding"):
        import torch
        self.torch = torch
        self.dims = dims
        self.dev = torch.device(device)
        self._keep = []
        up = self._upload
        self.desc = ModelDesc(dims.n_layers, dims.d_model, dims.n_heads, dims.n_kv_heads,
                              dims.head_dim, dims.ffn_dim, dims.vocab, dims.rope_theta,
                              dims.norm_eps)
        self.lim = Limits(max_batch, max_seq, max_tree, max_prompt)
        layers = (LayerWeights * dims.n_layers)()
        for l, lw in enumerate(target["layers"]):
            layers[l] = self._layer(lw)
        self._layers = layers
        self.tw = TargetWeights(up(target["embed"]), layers, up(target["final_norm"]),
                                up(target["lm_head"]))
        self.dw = DraftWeights(up(draft["fc"]), self._layer(draft["layer"]))
        tkv, dkv, ws, pw = msd_buffer_sizes(self.desc, self.lim)
        self.bufs_t = [torch.empty(n, dtype=torch.uint8, device=self.dev)
                       for n in (tkv, tkv, dkv, dkv, ws, pw)]
        self.bufs = Buffers(*[b.data_ptr() for b in self.bufs_t])
        self.stream = torch.cuda.current_stream(self.dev).cuda_stream
        self.ctx = msd_create(self.desc, self.lim, self.tw, self.dw, self.bufs, self.stream)
        self.set_draft_input(visual_input)

    def set_draft_input(self, visual_input):
        """Draft input of the visual prompt rows of later prefills: "embedding"
        (the method) or "feature" (the Visual Feature variant)."""
        msd_set_draft_input(self.ctx, DRAFT_VISUAL_INPUTS[visual_input])

    def use_caller_weights(self, enable=True):
        """Prompt products read the row-major target weights this engine
        uploaded (it keeps them until it is closed) instead of unpacking the
        packed copies."""
        msd_use_caller_weights(self.ctx, enable)

    def train_accumulate(self, seq, tokens, is_visual, visual_bits):
        """Gradient sums of one training sequence; returns its loss sums."""
        vis_t = None
        ptr = None
        if visual_bits is not None and len(visual_bits):
            vis_t = self.torch.from_numpy(np.ascontiguousarray(visual_bits).view(np.int16)).to(self.dev)
            ptr = vis_t.data_ptr()
        return msd_train_accumulate(self.ctx, seq, tokens, is_visual, ptr)

    def train_apply(self, lr):
        msd_train_apply(self.ctx, lr)

    def train_read(self, what):
        """{name: float32 numpy array} of the gradient sums (what 0) or the
        master parameters (what 1)."""
        shapes = train_param_shapes(self.dims)
        n = sum(int(np.prod(s)) for _, s in shapes)
        buf = self.torch.empty(n, dtype=self.torch.float32, device=self.dev)
        msd_train_read(self.ctx, what, buf.data_ptr(), n)
        flat = buf.cpu().numpy()
        out, o = {}, 0
        for name, s in shapes:
            k = int(np.prod(s))
            out[name] = flat[o:o + k].reshape(s)
            o += k
        return out

    def _upload(self, a):
        a = np.ascontiguousarray(a)
        t = self.torch.from_numpy(a.view(np.int16)).to(self.dev)
        self._keep.append(t)
        return t.data_ptr()

    def _layer(self, lw):
        u = self._upload
        return LayerWeights(u(lw["wq"]), u(lw["wk"]), u(lw["wv"]), u(lw["wo"]), u(lw["wg"]),
                            u(lw["wu"]), u(lw["wd"]), u(lw["attn_norm"]), u(lw["ffn_norm"]))

    def close(self):
        if self.ctx:
            msd_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # views of the caller-owned KV caches (bf16 bits as int16)
    def kv_views(self):
        d = self.dims
        B, S, hd, KV = self.lim.max_batch, self.lim.max_seq, d.head_dim, d.n_kv_heads
        tk = self.bufs_t[0].view(self.torch.int16).view(d.n_layers, B, KV, S, hd)
        tv = self.bufs_t[1].view(self.torch.int16).view(d.n_layers, B, KV, hd, S)
        dk = self.bufs_t[2].view(self.torch.int16).view(1, B, KV, S, hd)
        dv = self.bufs_t[3].view(self.torch.int16).view(1, B, KV, hd, S)
        return tk, tv, dk, dv

    def prefill(self, seq, tokens, is_visual, visual_bits):
        vis_t = None
        ptr = None
        if visual_bits is not None and len(visual_bits):
            vis_t = self.torch.from_numpy(np.ascontiguousarray(visual_bits).view(np.int16)).to(self.dev)
            ptr = vis_t.data_ptr()
        first = msd_prefill(self.ctx, seq, tokens, is_visual, ptr)
        return first

    def new_trees(self, n_seq):
        return self.torch.zeros(n_seq * ctypes.sizeof(Tree), dtype=self.torch.uint8, device=self.dev)

    @staticmethod
    def trees_to_host(trees_t, n_seq):
        raw = trees_t.cpu().numpy().tobytes()
        sz = ctypes.sizeof(Tree)
        return [Tree.from_buffer_copy(raw[i * sz:(i + 1) * sz]) for i in range(n_seq)]

    def draft_tree(self, seqs, spec, trees_t):
        msd_draft_tree(self.ctx, seqs, spec, trees_t.data_ptr())

    def verify(self, seqs, trees_t, n_nodes, want_logits=False):
        torch = self.torch
        amax = torch.empty(len(seqs) * n_nodes, dtype=torch.int32, device=self.dev)
        logits = None
        if want_logits:
            logits = torch.empty(len(seqs) * n_nodes, self.dims.vocab, dtype=torch.float32,
                                 device=self.dev)
        msd_verify(self.ctx, seqs, trees_t.data_ptr(), n_nodes, amax.data_ptr(),
                   logits.data_ptr() if logits is not None else None)
        return amax, logits

    def accept(self, seqs, trees_t, n_nodes, amax, want_slots=False):
        slots = None
        if want_slots:
            slots = self.torch.empty(len(seqs) * MAX_TREE, dtype=self.torch.int32, device=self.dev)
        em = msd_accept_compact(self.ctx, seqs, trees_t.data_ptr(), n_nodes, amax.data_ptr(),
                                slots.data_ptr() if slots is not None else None)
        return em, slots

    def accept_sample(self, seqs, trees_t, n_nodes, logits, temperature, seed,
                      want_slots=False):
        """Acceptance by speculative sampling; logits: verify's float32 logits."""
        slots = None
        if want_slots:
            slots = self.torch.empty(len(seqs) * MAX_TREE, dtype=self.torch.int32, device=self.dev)
        em = msd_accept_sample(self.ctx, seqs, trees_t.data_ptr(), n_nodes, logits.data_ptr(),
                               temperature, seed,
                               slots.data_ptr() if slots is not None else None)
        return em, slots

    def generate(self, seq, prompt, spec, n_new, record=False, temperature=0.0, seed=0):
        """Speculative decoding of one sequence: n_new tokens, greedy at
        temperature 0, else speculative sampling (the first token, from the
        prompt, is the greedy one either way)."""
        tokens, is_visual, visual = prompt
        out = [self.prefill(seq, tokens, is_visual, visual)]
        T = spec.n_nodes + 1
        trees = self.new_trees(1)
        cycles = []
        while len(out) < n_new:
            self.draft_tree([seq], spec, trees)
            amax, logits = self.verify([seq], trees, T, want_logits=temperature > 0)
            if temperature > 0:
                em, _ = self.accept_sample([seq], trees, T, logits, temperature, seed)
            else:
                em, _ = self.accept([seq], trees, T, amax)
            out.extend(int(t) for t in em[0])
            cycles.append(len(em[0]))
        return out[:n_new], cycles
