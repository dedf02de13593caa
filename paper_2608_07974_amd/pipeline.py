"""K chunks on one GPU as a ZeroLock stage pipeline with early forwarding
(libzl's zl_pipeline: event-bound hidden-state entries, in-flight depth,
update windows).  torch supplies device memory and one stream per stage;
every step runs in libzl."""
import torch

from . import zl
from .chunk import TorchChunk, check_batch, current_stream


class Pipeline:
    def __init__(self, cfgs, window=1, depth=2, device="cuda", head=None):
        """cfgs: one zl_config per stage (same d_model, dtype, max_batch,
        max_seq).  head: shared frozen (head_w, head_norm_w, head_norm_b)
        tensors, else the first chunk's are shared with the others."""
        zl.load()
        dev = torch.device(device)
        self.chunks = []
        for cfg in cfgs:
            ch = TorchChunk(cfg, device=dev, head=head)
            if head is None:
                head = (ch.head_w, ch.head_norm_w, ch.head_norm_b)
            self.chunks.append(ch)
        self.K = len(cfgs)
        self.window, self.depth = window, depth
        self.streams = [torch.cuda.Stream(device=dev) for _ in range(self.K)]
        nbytes = zl.zl_pipeline_entry_bytes(self.chunks[0].handle, self.K, depth)
        self._entries = torch.empty(nbytes + 256, dtype=torch.uint8, device=dev)
        base = (self._entries.data_ptr() + 255) // 256 * 256
        # the chunks' parameters were written on the current stream
        torch.cuda.current_stream(dev).synchronize()
        self.handle = zl.zl_pipeline_create([c.handle for c in self.chunks],
                                            [s.cuda_stream for s in self.streams],
                                            window, depth, base, nbytes)
        self.dtype = self.chunks[0].dtype

    def submit(self, h0, labels, pos_ids=None, seq_lens=None, losses=None):
        """Queue one micro-batch through all stages; returns (mb, losses[K])."""
        c0 = self.chunks[0]
        if labels is None:
            raise ValueError("labels are required")
        check_batch(self.dtype, c0.cfg.d_model, c0.device, h0, seq_lens, pos_ids, labels,
                    max_batch=c0.cfg.max_batch, max_seq=c0.cfg.max_seq)
        B, S, _ = h0.shape
        if losses is None:
            losses = torch.zeros(self.K, dtype=torch.float32, device=h0.device)
        elif (losses.dtype != torch.float32 or not losses.is_contiguous()
              or losses.numel() < self.K or losses.device != h0.device):
            raise ValueError(f"losses must be a contiguous float32 tensor of {self.K} elements "
                             f"on {h0.device}")
        # stage 0 copies its inputs on its own stream: order it after the
        # caller's stream (the inputs were produced there)
        ev = torch.cuda.Event()
        ev.record()
        self.streams[0].wait_event(ev)
        for s in self.streams:
            s.wait_event(ev)  # the losses buffer and outputs of earlier work
        p = lambda t: 0 if t is None else t.data_ptr()
        mb = zl.zl_pipeline_submit(self.handle, p(h0), p(labels), p(pos_ids), p(seq_lens), B, S,
                                   losses.data_ptr())
        return mb, losses

    def output(self, mb, shape):
        """The last stage's output of micro-batch mb, copied (on the caller's
        current stream, after the stage has written it) into a new tensor."""
        out = torch.empty(shape, dtype=self.dtype, device=self.chunks[0].device)
        zl.zl_pipeline_read_output(self.handle, mb, out.data_ptr(), current_stream())
        return out

    def sync(self):
        zl.zl_pipeline_sync(self.handle)

    def progress(self):
        return zl.zl_pipeline_progress(self.handle)

    def checkpoint(self, stage, path):
        zl.zl_pipeline_checkpoint(self.handle, stage, path)

    def close(self):
        if getattr(self, "handle", None):
            zl.zl_pipeline_destroy(self.handle)
            self.handle = None
        for c in self.chunks:
            c.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
