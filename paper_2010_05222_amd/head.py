"""Torch-facing wrapper of one class shard's PFC head step.

Allocates the step's output buffers and workspace once (torch device memory)
and calls the three C-ABI entry points on torch's current stream.  It does no
arithmetic of its own: sampling, forward, backward and the update all run in
libpfc's HIP kernels.
"""

import torch

from . import pfc as abi

DTYPES = {
    "f32": (torch.float32, abi.PFC_F32),
    "bf16": (torch.bfloat16, abi.PFC_BF16),
    "f16": (torch.float16, abi.PFC_F16),
}
MARGINS = {"cosface": abi.PFC_COSFACE, "arcface": abi.PFC_ARCFACE}


def _ptr(t):
    return 0 if t is None else t.data_ptr()


def _require(t, dtype, shape, name, device):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} contiguous={t.is_contiguous()}")
    if t.device != device:
        raise ValueError(f"{name}: expected device {device}, got {t.device}")


class PfcShard:
    """One GPU's class shard [class_offset, class_offset + C) of a PFC head.

    tau: threshold of the PFC* conflict filter (a negative logit whose
    unmargined cosine exceeds tau leaves the row's denominator); None, or any
    tau >= 1, is plain PFC.
    """

    def __init__(self, B, d, C, r, dtype="bf16", class_offset=0, s=64.0, m=0.5,
                 margin="arcface", lr=0.1, mu=0.9, device="cuda:0", tau=None):
        self.B, self.d, self.C, self.r = int(B), int(d), int(C), float(r)
        self.class_offset = int(class_offset)
        self.dtype_name = dtype
        self.tdtype, self.code = DTYPES[dtype]
        self.s, self.m, self.margin = float(s), float(m), MARGINS[margin]
        self.lr, self.mu = float(lr), float(mu)
        self.tau = None if tau is None else float(tau)
        self.device = torch.device(device)
        self.ws_bytes, self.cap = abi.pfc_workspace_bytes(self.B, self.d, self.C, self.r, self.code)
        dev = self.device
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.active = torch.empty(self.cap, dtype=torch.int32, device=dev)
        self.n_active = torch.empty(1, dtype=torch.int32, device=dev)
        self.labels_mapped = torch.empty(self.B, dtype=torch.int32, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.row_lse = torch.empty(self.B, dtype=torch.float32, device=dev)
        self.dX = torch.empty((self.B, self.d), dtype=torch.float32, device=dev)

    def _stream(self):
        return torch.cuda.current_stream(self.device).cuda_stream

    def sample(self, labels, seed):
        _require(labels, torch.int64, (self.B,), "labels", self.device)
        abi.pfc_sample(_ptr(labels), self.B, self.C, self.class_offset, self.r, int(seed),
                       _ptr(self.active), self.cap, _ptr(self.n_active), _ptr(self.labels_mapped),
                       _ptr(self.ws), self.ws_bytes, self._stream())

    def forward(self, X, W):
        _require(X, self.tdtype, (self.B, self.d), "X", self.device)
        _require(W, self.tdtype, (self.C, self.d), "W", self.device)
        abi.pfc_forward_loss(_ptr(X), self.code, self.B, self.d, _ptr(W), self.code, self.C,
                             _ptr(self.active), _ptr(self.n_active), self.cap,
                             _ptr(self.labels_mapped), self.code, self.s, self.m, self.margin,
                             2.0 if self.tau is None else self.tau, _ptr(self.loss),
                             _ptr(self.row_lse), _ptr(self.ws), self.ws_bytes, self._stream())

    def backward(self, X, W, M, W_master=None, row_lse=None):
        _require(X, self.tdtype, (self.B, self.d), "X", self.device)
        _require(W, self.tdtype, (self.C, self.d), "W", self.device)
        _require(M, torch.float32, (self.C, self.d), "momentum", self.device)
        if W_master is not None:
            _require(W_master, torch.float32, (self.C, self.d), "W_master", self.device)
        lse = self.row_lse if row_lse is None else row_lse
        abi.pfc_backward_update(_ptr(X), self.code, self.B, self.d, _ptr(W), self.code,
                                _ptr(W_master), _ptr(M), self.C, _ptr(self.active),
                                _ptr(self.n_active), self.cap, _ptr(self.labels_mapped),
                                self.code, self.s, self.m, self.margin, _ptr(lse), self.lr,
                                self.mu, _ptr(self.dX), _ptr(self.ws), self.ws_bytes,
                                self._stream())

    def step(self, X, labels, W, M, seed, W_master=None):
        """Sample, forward, backward and update of one mini-batch (all enqueued)."""
        self.sample(labels, seed)
        self.forward(X, W)
        self.backward(X, W, M, W_master)


class PfcPipeline:
    """A training loop's steps on one resident shard, with each step's
    sampling moved off the critical path: the active set of step t+1 depends
    only on its labels and seed, so it is drawn on a side stream while step t
    runs, into the second of two sets of step buffers (active set, mapped
    labels, outputs and workspace).  Results are those of PfcShard.step, bit
    for bit.

        pipe = PfcPipeline(B, d, C, r, ...)
        pipe.begin(labels[0], seeds[0])
        for t in range(T):
            out = pipe.step(X[t], W, M, labels[t + 1] if t + 1 < T else None,
                            seeds[t + 1] if t + 1 < T else None)
            # out.loss, out.row_lse, out.dX belong to step t (valid on the
            # current stream until step t + 2)
    """

    def __init__(self, B, d, C, r, **kw):
        self.parts = [PfcShard(B, d, C, r, **kw) for _ in range(2)]
        self.device = self.parts[0].device
        self.side = torch.cuda.Stream(device=self.device)
        self.done = [None, None]    # event: the last step that used each buffer set
        self.ready = [False, False]
        self.pending = [None, None]  # event: sampling into each buffer set
        self.t = 0

    def _sample(self, k, labels, seed):
        main = torch.cuda.current_stream(self.device)
        mark = torch.cuda.Event()
        mark.record(main)                     # the labels were made on the current stream
        self.side.wait_event(mark)
        if self.done[k] is not None:
            self.side.wait_event(self.done[k])
        with torch.cuda.stream(self.side):
            self.parts[k].sample(labels, seed)
        labels.record_stream(self.side)
        ev = torch.cuda.Event()
        ev.record(self.side)
        self.pending[k] = ev
        self.ready[k] = True

    def begin(self, labels, seed):
        """Draws the active set of the first step."""
        self.t = 0
        self.ready = [False, False]
        self._sample(0, labels, seed)

    def step(self, X, W, M, labels_next=None, seed_next=None, W_master=None):
        """Step t on the current stream (its sampling was drawn by the previous
        call, or by begin()); step t+1's sampling is drawn beside it."""
        a, b = self.t % 2, (self.t + 1) % 2
        if not self.ready[a]:
            raise RuntimeError("PfcPipeline.step: no active set drawn (call begin(), and pass "
                               "the next step's labels to every step but the last)")
        self.ready[a] = False
        main = torch.cuda.current_stream(self.device)
        main.wait_event(self.pending[a])
        if labels_next is not None:
            self._sample(b, labels_next, seed_next)
        cur = self.parts[a]
        cur.forward(X, W)
        cur.backward(X, W, M, W_master)
        ev = torch.cuda.Event()
        ev.record(main)
        self.done[a] = ev
        self.t += 1
        return cur


class TieredShard:
    """A class shard whose bank lives in pinned host memory (Sec. 3.3.3, the
    paragraph on asynchronous hierarchical class storage, Fig. async_pipeline).

    The bank - W in the storage dtype, fp32 momentum, and an fp32 master when
    `master` - holds all C rows (`W_bank`, `M_bank`, `P_bank`: pinned host
    tensors the caller fills).  Each step runs on a device slot of `cap` rows
    holding only its active rows; `n_slots` slots (2 or 3) are used in turn.
    While step t runs on its slot (current stream), an upload stream samples
    step t+1; after step t it stages the cold rows of S(t+1) into the next
    slot.  Rows that S(t+1) shares with S(t) (and, with three slots, with
    S(t-1)) are patched from those slots once their steps have updated them,
    and a download stream writes each slot back to the bank after its step.
    HIP events order the three streams:
      upload(t+1)   after download(t+1-n_slots)  (the slot and its id lists are
                    free, and every bank row it may read is current); its
                    sampling and patch(t-1 -> t+1) beside step t, its stage
                    and patch(t -> t+1) after step t (the newest copy wins)
      download(t)   after step t and the sampling of step t+1, whose rows it
                    leaves to download(t+1)
      step t+1      after its stage and patches
    With three slots the upload of step t+1 need not wait for the download of
    step t-1, so the two directions of the host link run at once.  Every copy
    is a libpfc kernel.

        ts = TieredShard(B, d, C, r, ...)
        ts.W_bank.copy_(W0); ts.M_bank.zero_()
        ts.begin(labels[0], seeds[0])
        for t in range(T):
            out = ts.step(X[t], labels[t + 1] if t + 1 < T else None, seeds[t + 1] ...)
            # out.loss, out.row_lse, out.dX belong to step t (valid on the
            # current stream until step t + n_slots)
        ts.finish()          # the bank holds every update
        ts.stale_rows()      # 0 unless a cold row was staged before its write-back
    """

    def __init__(self, B, d, C, r, dtype="bf16", class_offset=0, s=64.0, m=0.5,
                 margin="arcface", lr=0.1, mu=0.9, device="cuda:0", tau=None, master=False,
                 n_slots=3):
        if n_slots not in (2, 3):
            raise ValueError("n_slots must be 2 or 3")
        kw = dict(dtype=dtype, class_offset=class_offset, s=s, m=m, margin=margin, lr=lr, mu=mu,
                  device=device, tau=tau)
        self.n = int(n_slots)
        self.parts = [PfcShard(B, d, C, r, **kw) for _ in range(self.n)]
        p = self.parts[0]
        self.B, self.d, self.C, self.cap, self.device = p.B, p.d, p.C, p.cap, p.device
        dev, cap = self.device, self.cap
        self.W_bank = torch.empty((C, d), dtype=p.tdtype, pin_memory=True)
        self.M_bank = torch.zeros((C, d), dtype=torch.float32, pin_memory=True)
        self.P_bank = torch.empty((C, d), dtype=torch.float32, pin_memory=True) if master else None
        self.bank_version = torch.zeros(C, dtype=torch.int32, pin_memory=True)
        self.row_version = torch.zeros(C, dtype=torch.int32, device=dev)
        self.stale = torch.zeros(1, dtype=torch.int32, device=dev)
        self.slots = []
        for _ in range(self.n):
            sl = {"W": torch.empty((cap, d), dtype=p.tdtype, device=dev),
                  "M": torch.empty((cap, d), dtype=torch.float32, device=dev)}
            if master:
                sl["P"] = torch.empty((cap, d), dtype=torch.float32, device=dev)
            self.slots.append(sl)
        self.banks = {"W": self.W_bank, "M": self.M_bank}
        if master:
            self.banks["P"] = self.P_bank
        self.iota = torch.arange(cap, dtype=torch.int32, device=dev)
        self.up = torch.cuda.Stream(device=dev)
        self.down = torch.cuda.Stream(device=dev)
        self.ready = [torch.cuda.Event() for _ in range(self.n)]
        self.written = [None] * self.n      # event: last download of each slot
        self.staged = [False] * self.n
        self.t = 0

    def _row_bytes(self, key):
        return self.d * self.banks[key].element_size()

    def _keys(self, slot):
        return [k for k in ("M", "P", "W") if k in slot]

    def _stage(self, nxt, prevs, slot, version):
        # One launch moves the cold rows of every array; it checks and stamps
        # the versions.
        pv = [(_ptr(q.active), _ptr(q.n_active)) for q in prevs] + [(0, 0)] * (2 - len(prevs))
        keys = self._keys(slot)
        abi.pfc_bank_stage([_ptr(self.banks[k]) for k in keys], [_ptr(slot[k]) for k in keys],
                           [self._row_bytes(k) for k in keys], self.C, _ptr(nxt.active),
                           _ptr(nxt.n_active), pv[0][0], pv[0][1], pv[1][0], pv[1][1], self.cap,
                           _ptr(self.bank_version), _ptr(self.row_version), version,
                           _ptr(self.stale), self.up.cuda_stream)

    def _patch(self, prv, src, nxt, dst):
        keys = self._keys(src)
        abi.pfc_bank_patch([_ptr(src[k]) for k in keys], [_ptr(dst[k]) for k in keys],
                           [self._row_bytes(k) for k in keys], _ptr(prv.active),
                           _ptr(prv.n_active), _ptr(nxt.active), _ptr(nxt.n_active), self.cap,
                           self.up.cuda_stream)

    def _writeback(self, part, slot, version, nxt):
        # One launch writes every array's rows back; a row's version is
        # stamped after all of its arrays have reached the bank.  Rows the
        # next step holds are left to its write-back.
        na, nn = (_ptr(nxt.active), _ptr(nxt.n_active)) if nxt else (0, 0)
        keys = self._keys(slot)
        abi.pfc_bank_writeback([_ptr(slot[k]) for k in keys], [_ptr(self.banks[k]) for k in keys],
                               [self._row_bytes(k) for k in keys], _ptr(part.active),
                               _ptr(part.n_active), na, nn, self.cap, self.C,
                               _ptr(self.bank_version), version, self.down.cuda_stream)

    def _run_step(self, part, X, slot):
        _require(X, part.tdtype, (self.B, self.d), "X", self.device)
        stream = torch.cuda.current_stream(self.device).cuda_stream
        tau = 2.0 if part.tau is None else part.tau
        abi.pfc_forward_loss(_ptr(X), part.code, self.B, self.d, _ptr(slot["W"]), part.code,
                             self.C, _ptr(self.iota), _ptr(part.n_active), self.cap,
                             _ptr(part.labels_mapped), part.code, part.s, part.m, part.margin,
                             tau, _ptr(part.loss), _ptr(part.row_lse), _ptr(part.ws),
                             part.ws_bytes, stream)
        abi.pfc_backward_update(_ptr(X), part.code, self.B, self.d, _ptr(slot["W"]), part.code,
                                _ptr(slot.get("P")), _ptr(slot["M"]), self.C, _ptr(self.iota),
                                _ptr(part.n_active), self.cap, _ptr(part.labels_mapped),
                                part.code, part.s, part.m, part.margin, _ptr(part.row_lse),
                                part.lr, part.mu, _ptr(part.dX), _ptr(part.ws), part.ws_bytes,
                                stream)

    def _mark_main(self):
        ev = torch.cuda.Event()
        ev.record(torch.cuda.current_stream(self.device))
        return ev

    def _sample_into(self, k, labels, seed):
        """Sample a step into parts[k] on the upload stream, once slot k is free."""
        self.up.wait_event(self._mark_main())          # labels were made on the current stream
        if self.written[k] is not None:
            self.up.wait_event(self.written[k])
        sampled = torch.cuda.Event()
        with torch.cuda.stream(self.up):
            self.parts[k].sample(labels, seed)
            sampled.record(self.up)
        labels.record_stream(self.up)
        return sampled

    def begin(self, labels, seed):
        """Samples step 0 and stages all of its rows."""
        self.t = 0
        self._sample_into(0, labels, seed)
        self._stage(self.parts[0], [], self.slots[0], 1)
        self.ready[0].record(self.up)
        self.staged = [False] * self.n
        self.staged[0] = True

    def step(self, X, labels_next=None, seed_next=None):
        """Step t on the current stream; step t+1's rows are staged alongside."""
        t, n = self.t, self.n
        a, b, z = t % n, (t + 1) % n, (t - 1) % n
        cur, nxt = self.parts[a], self.parts[b]
        if not self.staged[a]:
            raise RuntimeError("TieredShard.step: no staged rows (call begin(), and pass the "
                               "next step's labels to every step but the last)")
        self.staged[a] = False
        older = self.parts[z] if (n >= 3 and t >= 1) else None
        sampled = None
        if labels_next is not None:
            sampled = self._sample_into(b, labels_next, seed_next)
            if older:
                # Step t-1 is done: the upload stream waited for it before the
                # previous patch.
                self._patch(older, self.slots[z], nxt, self.slots[b])
        main = torch.cuda.current_stream(self.device)
        main.wait_event(self.ready[a])
        self._run_step(cur, X, self.slots[a])
        done = self._mark_main()
        if labels_next is not None:
            # The cold rows go up after the step: a copy kernel beside the
            # step's kernels finds few free CUs and moves little, while it
            # slows them down.
            self.up.wait_event(done)
            self._stage(nxt, [cur] + ([older] if older else []), self.slots[b], t + 2)
            self._patch(cur, self.slots[a], nxt, self.slots[b])
            self.ready[b].record(self.up)
            self.staged[b] = True
        self.down.wait_event(done)
        if sampled is not None:
            self.down.wait_event(sampled)
        self._writeback(cur, self.slots[a], t + 1, nxt if sampled is not None else None)
        ev = torch.cuda.Event()
        ev.record(self.down)
        self.written[a] = ev
        self.t += 1
        return cur

    def finish(self):
        """The current stream waits for every staging and write-back."""
        main = torch.cuda.current_stream(self.device)
        main.wait_stream(self.up)
        main.wait_stream(self.down)

    def stale_rows(self):
        """Rows staged from the bank before their last update was written back
        (or with an id outside the shard); synchronises."""
        self.finish()
        return int(self.stale.item())
