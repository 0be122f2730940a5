"""MI355X (gfx950) implementation of one pipelined-gradient-coding step.

The computation lives in libpgc.so (C ABI: include/pgc.h; HIP kernels in
csrc/).  `_lib` binds every entry point by name; `PGCSession` is plumbing that
lets torch own the workspace memory and the stream.  There is no fallback:
if the library is missing, every call raises.
"""

from ._lib import *  # noqa: F401,F403  (the C entry points, same names)
from . import _lib


class PGCSession:
    """A configured PGC context bound to a torch-allocated workspace on one GPU.

    scheme: "FR", "CR", "CR_REAL" or "IS_SGD"; model: "logistic", "lsq" or "mlp".
    pipelined=False runs gradient coding instead (every slot evaluated each step).
    q (the parameter length) follows from the model shape.
    """

    def __init__(self, scheme, n, c, model, N, d_in, hidden=0, classes=0, code_seed=0,
                 device="cuda", stream=None, pipelined=True):
        import torch
        self.n, self.c, self.N, self.d_in = int(n), int(c), int(N), int(d_in)
        self.scheme, self.model = scheme, model
        if model == "mlp":
            self.q = d_in * hidden + hidden + hidden * classes + classes
        else:
            self.q = int(d_in)
        self.device = torch.device(device)
        if self.device.type == "cuda" and self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.ctx = _lib.pgc_init(scheme, n, c, self.q)
        try:
            _lib.pgc_configure(self.ctx, model, N, d_in, hidden, classes, code_seed)
            nbytes = _lib.pgc_workspace_bytes(self.ctx)
            self.workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=self.device)
            if stream is None:
                stream = torch.cuda.current_stream(self.device).cuda_stream
            _lib.pgc_set_stream(self.ctx, stream)
            _lib.pgc_bind_workspace(self.ctx, self.workspace, nbytes)
        except Exception:
            _lib.pgc_destroy(self.ctx)
            self.ctx = None
            raise
        self.n_coded = _lib.pgc_num_coded(self.ctx)
        if not pipelined:
            _lib.pgc_set_pipelining(self.ctx, False)

    def step(self, X, y, w, straggler_mask, lr):
        """One step; X, y, w are GPU tensors holding at least N*d_in, N and q elements."""
        self._check_step_args(X, y, w)
        _lib.pgc_step(self.ctx, X, y, w, straggler_mask, lr, self.n)

    def _check_step_args(self, X, y, w):
        import torch
        x_dtype = torch.bfloat16 if self.model == "mlp" else torch.float32
        y_dtype = torch.int32 if self.model == "mlp" else torch.float32
        for name, t, dtype, numel in (("X", X, x_dtype, self.N * self.d_in), ("y", y, y_dtype, self.N),
                                      ("w", w, torch.float32, self.q)):
            if t.dtype != dtype or t.numel() < numel or not t.is_contiguous() or t.device != self.device:
                raise ValueError("%s must be a contiguous %s tensor of >= %d elements on %s"
                                 % (name, dtype, numel, self.device))

    def step_noalloc(self, X, y, w, straggler_mask, lr):
        """The same step through pgc_step_noalloc (linear models; partial sums in
        the library's fixed device array)."""
        self._check_step_args(X, y, w)
        _lib.pgc_step_noalloc(self.ctx, X, y, w, straggler_mask, lr, self.n)

    def restart(self):
        """Start over at t = 0 (the warm-up step) by binding the workspace again;
        the next step refills the whole ring."""
        _lib.pgc_bind_workspace(self.ctx, self.workspace, _lib.pgc_workspace_bytes(self.ctx))

    def save_state(self):
        """The pipeline state (step counter and gradient ring) in a new uint8 GPU
        tensor, filled on the session's stream."""
        import torch
        out = torch.empty(_lib.pgc_state_bytes(self.ctx), dtype=torch.uint8, device=self.device)
        _lib.pgc_save_state(self.ctx, out)
        return out

    def load_state(self, state):
        """Resume from a state saved by a session of the same configuration."""
        _lib.pgc_load_state(self.ctx, state)

    def set_stream(self, stream):
        """Launch later steps on `stream` (a torch.cuda.Stream or a raw HIP stream handle)."""
        handle = getattr(stream, "cuda_stream", stream)
        _lib.pgc_set_stream(self.ctx, handle)

    @property
    def t(self):
        return _lib.pgc_get_step(self.ctx)

    def decode_coeffs(self, straggler_mask):
        return _lib.pgc_decode_coeffs(self.ctx, straggler_mask, self.n)

    def placement(self):
        return _lib.pgc_placement(self.ctx, self.n, self.c)

    def schedule(self, t):
        return _lib.pgc_schedule(self.ctx, t, self.n)

    def encoding_matrix(self):
        return _lib.pgc_encoding_matrix(self.ctx, self.n)

    def _vec(self):
        import torch
        return torch.empty(self.q, dtype=torch.float32, device=self.device)

    def ring(self, worker, slot):
        out = self._vec()
        _lib.pgc_read_ring(self.ctx, worker, slot, out)
        return out

    def coded(self, index):
        out = self._vec()
        _lib.pgc_read_coded(self.ctx, index, out)
        return out

    def decoded(self):
        out = self._vec()
        _lib.pgc_read_decoded(self.ctx, out)
        return out

    def close(self):
        if self.ctx is not None:
            _lib.pgc_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
