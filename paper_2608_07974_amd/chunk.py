"""A chunk whose buffers live in torch device tensors.

torch provides device memory and the current HIP stream; every step of the
update runs in libzl's kernels through the C ABI (zl.py).  Parameter keys
are "L{layer}.{name}" with the names of zl_param_layout.
"""
import numpy as np
import torch

from . import zl

_TORCH_DT = {zl.ZL_F32: torch.float32, zl.ZL_BF16: torch.bfloat16}


def _ptr(t):
    return 0 if t is None else t.data_ptr()


def current_stream():
    return torch.cuda.current_stream().cuda_stream


def _norm_device(device):
    """torch.device with the index filled in ("cuda" -> the current GPU)."""
    device = torch.device(device)
    if device.type == "cuda" and device.index is None:
        device = torch.device("cuda", torch.cuda.current_device())
    return device


def _check_int_tensor(name, t, device, numel):
    if t.dtype != torch.int32 or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous int32 tensor")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, not {t.device}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements, not {t.numel()}")


def check_batch(dtype, d_model, device, h_in, seq_lens=None, pos_ids=None, labels=None,
                h_out=None, max_batch=None, max_seq=None):
    """Raises before any pointer reaches libzl when a tensor does not match
    what the kernels read: h_in a contiguous [B, S, d_model] tensor of the
    chunk's dtype on `device`; seq_lens B, pos_ids and labels B*S int32
    elements on the same device; h_out like h_in.  The kernels index these
    buffers by B and S alone, so a short or host-side tensor would be read
    out of bounds on the GPU."""
    device = _norm_device(device)
    if h_in.dtype != dtype or not h_in.is_contiguous() or h_in.dim() != 3:
        raise TypeError(f"h_in must be a contiguous [B, S, d] {dtype} tensor")
    if h_in.device != device:
        raise ValueError(f"h_in must be on {device}, not {h_in.device}")
    B, S, d = h_in.shape
    if d != d_model:
        raise ValueError(f"h_in's last dimension is {d}, the chunk's d_model is {d_model}")
    if B < 1 or S < 1 or (max_batch is not None and B > max_batch) or \
            (max_seq is not None and S > max_seq):
        raise ValueError(f"B = {B}, S = {S} outside [1, {max_batch}] x [1, {max_seq}]")
    for name, t, n in (("seq_lens", seq_lens, B), ("pos_ids", pos_ids, B * S),
                       ("labels", labels, B * S)):
        if t is not None:
            _check_int_tensor(name, t, device, n)
    if h_out is not None:
        if h_out.dtype != dtype or h_out.shape != h_in.shape or not h_out.is_contiguous():
            raise TypeError("h_out must match h_in in shape and dtype and be contiguous")
        if h_out.device != device:
            raise ValueError(f"h_out must be on {device}, not {h_out.device}")


def config_from_shape(shp, alpha=0.5, consis="reverse", optimizer="adamw", lr=1e-4, wd=0.01,
                      max_batch=None, max_seq=None):
    """zl_config for a workload shape (arch, widths, dtype) and objective."""
    return zl.make_config(
        zl.ZL_ARCH_LLAMA if shp.arch == "llama" else zl.ZL_ARCH_GPT2, shp.n_layers, shp.d_model,
        shp.n_heads, shp.n_kv_heads, shp.head_dim, shp.d_ff, shp.vocab, norm_eps=shp.norm_eps,
        rope_theta=max(shp.rope_theta, 2.0),
        dtype=zl.ZL_BF16 if shp.dtype == "bf16" else zl.ZL_F32, alpha=alpha,
        consis=zl.ZL_KL_REVERSE if consis == "reverse" else zl.ZL_KL_FORWARD,
        optimizer=zl.ZL_ADAMW if optimizer == "adamw" else zl.ZL_SGD, lr=lr, beta1=0.9,
        beta2=0.999, eps=1e-8, weight_decay=wd, max_batch=max_batch or shp.batch,
        max_seq=max_seq or shp.seq, adapter_rank=getattr(shp, "adapter_rank", 0),
        lora_rank=getattr(shp, "lora_rank", 0), lora_alpha=getattr(shp, "lora_alpha", 16.0))


class TorchChunk:
    """`head`: optional (head_w, head_norm_w, head_norm_b) device tensors to
    share with other chunks (the frozen head is read-only).  With LoRA
    (cfg.lora_rank > 0) the frozen base tensors sit in base_master /
    base_shadow and master holds the trainable factors (and adapter)."""

    def __init__(self, cfg, device="cuda", head=None):
        zl.load()
        self.cfg = cfg
        self.device = _norm_device(device)
        self.dtype = _TORCH_DT[cfg.dtype]
        self.n_params, self.layout = zl.zl_param_layout(cfg)
        dev = self.device
        n = self.n_params
        self.master = torch.zeros(n, dtype=torch.float32, device=dev)
        self.shadow = torch.zeros(n, dtype=torch.bfloat16, device=dev) if cfg.dtype == zl.ZL_BF16 else None
        self.grad = torch.zeros(n, dtype=torch.float32, device=dev)
        adam = cfg.optimizer == zl.ZL_ADAMW
        self.adam_m = torch.zeros(n, dtype=torch.float32, device=dev) if adam else None
        self.adam_v = torch.zeros(n, dtype=torch.float32, device=dev) if adam else None
        d, V = cfg.d_model, cfg.vocab
        if head is not None:
            self.head_w, self.head_norm_w, self.head_norm_b = head
        else:
            self.head_w = torch.zeros(V, d, dtype=self.dtype, device=dev)
            self.head_norm_w = torch.ones(d, dtype=torch.float32, device=dev)
            self.head_norm_b = (torch.zeros(d, dtype=torch.float32, device=dev)
                                if cfg.arch == zl.ZL_ARCH_GPT2 else None)
        self.base_master = self.base_shadow = None
        self.base_layout = []
        if cfg.lora_rank:
            nb, self.base_layout = zl.zl_param_layout(zl.base_config(cfg))
            self.base_master = torch.zeros(nb, dtype=torch.float32, device=dev)
            if cfg.dtype == zl.ZL_BF16:
                self.base_shadow = torch.zeros(nb, dtype=torch.bfloat16, device=dev)
        self.ws_bytes = zl.zl_workspace_size(cfg)
        self._ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=dev)
        self.ws_ptr = (self._ws.data_ptr() + 255) // 256 * 256
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        bufs = zl.zl_buffers(_ptr(self.master), _ptr(self.shadow), _ptr(self.grad),
                             _ptr(self.adam_m), _ptr(self.adam_v), _ptr(self.head_w),
                             _ptr(self.head_norm_w), _ptr(self.head_norm_b),
                             _ptr(self.base_master), _ptr(self.base_shadow))
        self.handle = zl.zl_chunk_create(cfg, bufs, self.ws_ptr, self.ws_bytes)
        self._tokens = None  # B*S of the last forward (labels must match it)
        self.by_key = {f"L{t['layer']}.{t['name']}": t for t in self.layout}
        self.base_by_key = {f"L{t['layer']}.{t['name']}": t for t in self.base_layout}

    def close(self):
        if self.handle:
            zl.zl_chunk_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------ params
    def view(self, buf, key):
        """A trainable tensor as stored (LoRA factors of a rank that is not a
        multiple of 8 include their zero padding)."""
        t = self.by_key[key]
        return buf[t["offset"]: t["offset"] + t["numel"]].view(*t["shape"])

    def logical(self, buf, key):
        """A trainable tensor at its configured shape (LoRA factors without
        their padding: A [r, in], B [out, r])."""
        v = self.view(buf, key)
        r = self.cfg.lora_rank
        if key.endswith("_la"):
            return v[:r]
        if key.endswith("_lb"):
            return v[:, :r]
        return v

    def padding(self, buf, key):
        """The padding of a stored LoRA factor (empty for other tensors)."""
        v = self.view(buf, key)
        r = self.cfg.lora_rank
        if key.endswith("_la"):
            return v[r:]
        if key.endswith("_lb"):
            return v[:, r:]
        return v[:0]

    def load_params(self, params):
        """Trainable tensors by key into master (at their configured shape;
        the padding of stored LoRA factors is zeroed by zl_refresh_shadow);
        with LoRA, frozen base tensors (keys of the base layout) into
        base_master."""
        for key, val in params.items():
            src = torch.as_tensor(np.asarray(val, np.float32))
            if key in self.by_key:
                self.logical(self.master, key).copy_(src)
            elif key in self.base_by_key:
                t = self.base_by_key[key]
                self.base_master[t["offset"]: t["offset"] + t["numel"]].view(*t["shape"]).copy_(src)
            else:
                raise KeyError(key)
        zl.zl_refresh_shadow(self.handle, current_stream())

    def load_head(self, head_w, head_norm_w, head_norm_b=None):
        self.head_w.copy_(torch.as_tensor(np.asarray(head_w, np.float32)).to(self.dtype))
        self.head_norm_w.copy_(torch.as_tensor(np.asarray(head_norm_w, np.float32)))
        if self.head_norm_b is not None and head_norm_b is not None:
            self.head_norm_b.copy_(torch.as_tensor(np.asarray(head_norm_b, np.float32)))

    def tensors(self, buf):
        """Every trainable tensor of `buf` at its configured shape, float64."""
        torch.cuda.synchronize(self.device)
        return {k: self.logical(buf, k).detach().cpu().double().numpy() for k in self.by_key}

    # ------------------------------------------------------------ update
    def _check_inputs(self, h_in, seq_lens=None, pos_ids=None, labels=None, h_out=None):
        check_batch(self.dtype, self.cfg.d_model, self.device, h_in, seq_lens, pos_ids, labels,
                    h_out, max_batch=self.cfg.max_batch, max_seq=self.cfg.max_seq)

    def forward(self, h_in, seq_lens=None, pos_ids=None, h_out=None):
        self._check_inputs(h_in, seq_lens, pos_ids, None, h_out)
        B, S, _ = h_in.shape
        self._tokens = B * S
        if h_out is None:
            h_out = torch.empty_like(h_in)
        zl.zl_chunk_forward(self.handle, _ptr(h_in), _ptr(seq_lens), _ptr(pos_ids), B, S,
                            _ptr(h_out), current_stream())
        return h_out

    def objective(self, labels):
        _check_int_tensor("labels", labels, self.device, None)
        if self._tokens is not None and labels.numel() != self._tokens:
            raise ValueError(f"labels must hold B*S = {self._tokens} elements")
        zl.zl_local_objective(self.handle, _ptr(labels), _ptr(self.loss), current_stream())
        return self.loss

    def backward(self, grad_scale=1.0, accumulate=0):
        zl.zl_chunk_backward(self.handle, grad_scale, accumulate, current_stream())

    def step(self):
        zl.zl_optimizer_step(self.handle, current_stream())

    def update(self, h_in, labels, seq_lens=None, pos_ids=None, h_out=None):
        self._check_inputs(h_in, seq_lens, pos_ids, labels, h_out)
        B, S, _ = h_in.shape
        if h_out is None:
            h_out = torch.empty_like(h_in)
        zl.zl_chunk_update(self.handle, _ptr(h_in), _ptr(seq_lens), _ptr(pos_ids), _ptr(labels),
                           B, S, _ptr(h_out), _ptr(self.loss), current_stream())
        return h_out

    def save(self, path, microbatches=0, windows=0):
        """Checkpoint parameters, optimizer state and step (after the stream's work)."""
        zl.zl_chunk_save(self.handle, path, microbatches, windows, current_stream())

    def restore(self, path):
        """Load a checkpoint; returns its (microbatches, windows) progress."""
        return zl.zl_chunk_load(self.handle, path, current_stream())

    def inspect_device(self, name, layer=0):
        """A workspace view as a [rows, cols] device tensor (no copy; valid
        until the next call that rewrites the workspace; read only)."""
        v = zl.zl_inspect(self.handle, name, layer)
        dt = torch.bfloat16 if v["dtype"] == zl.ZL_BF16 else torch.float32
        esz = 2 if dt == torch.bfloat16 else 4
        n = v["rows"] * v["ld"]
        # the workspace bytes at v["ptr"], through the owning tensor
        off = v["ptr"] - self._ws.data_ptr()
        if off < 0 or off + n * esz > self._ws.numel():
            raise ValueError(f"view {name} lies outside the workspace")
        src = self._ws[off: off + n * esz].view(dt)
        return src.view(v["rows"], v["ld"])[:, : v["cols"]]

    def inspect(self, name, layer=0):
        """Copy of a workspace view as a float64 numpy array."""
        t = self.inspect_device(name, layer)
        torch.cuda.synchronize(self.device)
        return t.double().cpu().numpy()
