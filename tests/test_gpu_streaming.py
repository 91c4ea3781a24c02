"""Weight streaming on the GPU (qg_run_layers): packed weights copied from
pinned host memory into device slots on a copy stream, overlapped with the
GEMMs. Only where the weight bytes come from changes, so every output must be
bit-identical to the run with all weights resident (the paper's claim for
streaming, Sec. 4, weight-streaming paragraph), for any slot count, any
resident subset and across consecutive steps. The resident run itself is
checked against the CPU oracle (every output of every layer within
|y - y_ref| <= 1e-3 sum|a w|), so the streamed runs are tied to the oracle,
not only to another run of the same kernels."""
import ctypes

import pytest
import torch

import oracle
import paper_2609_21849_amd as q
import synth
from gpu_util import DEV, check_linear, log, to_dev_bf16

pytestmark = pytest.mark.gpu

FP8, NV, MX, BF16 = q.QG_FMT_FP8_E4M3, q.QG_FMT_NVFP4, q.QG_FMT_MXFP4, q.QG_FMT_BF16
# (a_fmt, w_fmt, m, n, k, out dtype)
LAYERS = [(FP8, FP8, 256, 512, 768, q.QG_OUT_BF16), (NV, NV, 200, 768, 512, q.QG_OUT_BF16),
          (BF16, NV, 16, 1024, 512, q.QG_OUT_BF16), (MX, MX, 300, 512, 1024, q.QG_OUT_F32),
          (FP8, FP8, 512, 1024, 1024, q.QG_OUT_F32), (NV, NV, 64, 256, 1024, q.QG_OUT_BF16),
          (BF16, NV, 1, 3072, 1024, q.QG_OUT_BF16)]


class Model:
    def __init__(self):
        self.x, self.codes, self.bs, self.ts, self.wdev, self.whost, self.y = [], [], [], [], [], [], []
        self.x_bits, self.w_bits = [], []
        for i, (af, wf, m, n, k, od) in enumerate(LAYERS):
            self.x_bits.append(synth.normal_bf16(m, k, 1.0, 40 + i, 0))
            self.w_bits.append(synth.normal_bf16(n, k, 0.02, 40 + i, 1))
            x = to_dev_bf16(self.x_bits[-1])
            w = to_dev_bf16(self.w_bits[-1])
            packed = q.pack(q.quantize(w, wf))
            host = torch.empty(packed.numel(), dtype=torch.uint8, pin_memory=True)
            host.copy_(packed)
            if af == FP8:
                codes, bs = torch.empty((m, k), dtype=torch.uint8, device=DEV), None
            elif af == NV:
                codes, bs = (torch.empty((m, k // 2), dtype=torch.uint8, device=DEV),
                             torch.empty((m, k // 16), dtype=torch.uint8, device=DEV))
            elif af == MX:
                codes, bs = (torch.empty((m, k // 2), dtype=torch.uint8, device=DEV),
                             torch.empty((m, k // 32), dtype=torch.uint8, device=DEV))
            else:
                codes, bs = None, None
            ts = torch.empty(1, dtype=torch.float32, device=DEV) if af in (FP8, NV) else None
            y = torch.empty((m, n), dtype=torch.float32 if od == q.QG_OUT_F32 else torch.bfloat16, device=DEV)
            for lst, v in ((self.x, x), (self.codes, codes), (self.bs, bs), (self.ts, ts), (self.wdev, packed),
                           (self.whost, host), (self.y, y)):
                lst.append(v)
        torch.cuda.synchronize()
        self.slot_bytes = max(t.numel() for t in self.wdev)
        self.slot_bytes = (self.slot_bytes + 255) // 256 * 256

    def layers(self, resident):
        out = []
        for i, (af, wf, m, n, k, od) in enumerate(LAYERS):
            r = bool(resident[i])
            w = self.wdev[i] if r else self.whost[i]
            out.append(q.StreamLayer(x=self.x[i].data_ptr(), a_fmt=af,
                                     a_codes=self.codes[i].data_ptr() if self.codes[i] is not None else None,
                                     a_block_scales=self.bs[i].data_ptr() if self.bs[i] is not None else None,
                                     a_tensor_scale=self.ts[i].data_ptr() if self.ts[i] is not None else None,
                                     w_fmt=wf, w_packed=w.data_ptr(), w_packed_bytes=w.numel(), resident=int(r),
                                     m=m, n=n, k=k, y=self.y[i].data_ptr(), y_dtype=od))
        return out


def _events(n):
    evs = []
    for _ in range(n):
        e = torch.cuda.Event()
        e.record()          # creates the underlying event
        evs.append(e)
    return evs


@pytest.fixture(scope="module")
def model():
    return Model()


@pytest.fixture(scope="module")
def reference(model):
    cur = ctypes.c_int32(0)
    q.qg_run_layers(model.layers([1] * len(LAYERS)), [], 0, [], [], cur)
    torch.cuda.synchronize()
    ref = [y.clone() for y in model.y]
    # the same outputs as separate quantize + linear calls
    for i, (af, wf, m, n, k, od) in enumerate(LAYERS):
        a = model.x[i] if af == BF16 else q.quantize(model.x[i], af)
        y = q.linear(a, model.wdev[i], wf, n, out_dtype=od)
        torch.cuda.synchronize()
        assert torch.equal(y, ref[i]), i
    # and every output of the resident run against the oracle
    kinds = {(FP8, FP8): "fp8", (NV, NV): "nvfp4", (BF16, NV): "w4a16", (MX, MX): "mxfp4"}
    for i, (af, wf, m, n, k, od) in enumerate(LAYERS):
        r = oracle.linear_reference(kinds[(af, wf)], model.x_bits[i], model.w_bits[i])
        worst = check_linear(ref[i], r, name="streaming layer %d %s %dx%dx%d (every output)" % (i, kinds[(af, wf)], m, n, k))
        log("streaming layer %d %s %dx%dx%d max err/B %.3e" % (i, kinds[(af, wf)], m, n, k, worst))
    return ref


@pytest.mark.parametrize("n_slots", [1, 2, 3])
@pytest.mark.parametrize("pattern", ["all_streamed", "alternate", "first_resident"])
def test_streamed_outputs_are_bit_identical(model, reference, n_slots, pattern):
    n = len(LAYERS)
    resident = {"all_streamed": [0] * n, "alternate": [i % 2 for i in range(n)],
                "first_resident": [1 if i < 2 else 0 for i in range(n)]}[pattern]
    log("streaming slots=%d pattern=%s" % (n_slots, pattern))
    slots = [torch.empty(model.slot_bytes, dtype=torch.uint8, device=DEV) for _ in range(n_slots)]
    ready, free = _events(n_slots), _events(n_slots)
    copy_stream = torch.cuda.Stream()
    cur = ctypes.c_int32(0)
    streamed = n - sum(resident)
    for step in range(3):
        for y in model.y:
            y.zero_()
        q.qg_run_layers(model.layers(resident), slots, model.slot_bytes, [e.cuda_event for e in ready],
                        [e.cuda_event for e in free], cur, compute_stream=torch.cuda.current_stream(),
                        copy_stream=copy_stream)
        torch.cuda.synchronize()
        assert cur.value == (streamed * (step + 1)) % n_slots
        for i, (y, r) in enumerate(zip(model.y, reference)):
            assert torch.equal(y, r), "layer %d step %d" % (i, step)
