"""Several host threads call the library at the same time, each on a stream
of its own with buffers of its own (the library is documented as safe to
call from several host threads): every result must be bit-identical to the
same calls made one after another on one stream.  The ctypes calls release
the GIL, so the threads' validation, dispatch and launches overlap on the
host and their kernels overlap on the device."""

import threading

import numpy as np
import pytest
import torch

from paper_2609_04098_amd import linear as L
from paper_2609_04098_amd import synth
from tests.gpu_common import log, to_dev_bf16

pytestmark = pytest.mark.gpu

# (m, n, k, segment offsets): each case takes a different GEMM path.
CASES = [
    (513, 520, 1024, [0, 100, 520]),       # 256 x 256 tiles with scale super-stages
    (777, 1300, 384, [0, 500, 1300]),      # 256 x 256 tiles, K % 256 != 0, ragged M and N
    (300, 96, 5184, [0, 48, 96]),          # tall-skinny split-K
    (7, 4100, 1024, [0, 4000, 4100]),      # decode split-K; also the fused quantize + GEMM
]
REPS = 3


class Job:
    def __init__(self, i, m, n, k, offs):
        rng = np.random.default_rng(900 + i)
        x = rng.standard_normal((m, k))
        x[:, rng.choice(k, max(1, k // 200), replace=False)] *= 100.0
        w = rng.standard_normal((n, k)) * 0.02
        self.x = to_dev_bf16(synth.f64_to_bf16_bits(x))
        self.pw = L.pack_weight(to_dev_bf16(synth.f64_to_bf16_bits(w)), offs)
        dev = self.x.device
        self.aq = L.alloc_act(m, k, dev)
        self.aws = L.act_workspace(m, k, dev)
        self.gws = L.gemm_workspace(m, n, k, dev)
        self.y = torch.empty((m, n), dtype=torch.bfloat16, device=dev)
        self.fused = m <= 32
        if self.fused:
            self.fq = L.alloc_act(m, k, dev)
            self.fws = L.quantize_gemm_workspace(m, n, k, dev)
            self.fy = torch.empty((m, n), dtype=torch.bfloat16, device=dev)
        self.stream = torch.cuda.Stream()

    def outputs(self):
        out = [self.aq.codes, self.aq.scales, self.aq.g, self.y]
        if self.fused:
            out += [self.fq.codes, self.fq.scales, self.fq.g, self.fy]
        return out

    def run(self, stream):
        L.quantize_act(self.x, out=self.aq, workspace=self.aws, stream=stream)
        L.gemm(self.aq, self.pw, out=self.y, workspace=self.gws, stream=stream)
        if self.fused:
            L.quantize_gemm(self.x, self.pw, out=self.fy, act_out=self.fq, workspace=self.fws, stream=stream)


def test_concurrent_host_threads_match_serial_calls():
    jobs = [Job(i, *c) for i, c in enumerate(CASES)]
    for j in jobs:
        j.run(None)
    torch.cuda.synchronize()
    ref = [[t.clone() for t in j.outputs()] for j in jobs]

    for rep in range(REPS):
        for j in jobs:
            for t in j.outputs():
                t.fill_(0x7F if t.dtype == torch.uint8 else float("nan"))
        torch.cuda.synchronize()
        start = threading.Barrier(len(jobs))
        errors = []

        def work(j):
            try:
                start.wait()
                for _ in range(2):          # the second pass overwrites the first with the same bits
                    j.run(j.stream)
            except Exception as e:          # reported by the main thread
                errors.append(repr(e))

        threads = [threading.Thread(target=work, args=(j,)) for j in jobs]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=60)
        assert not any(t.is_alive() for t in threads), "a host thread did not finish"
        assert not errors, errors
        torch.cuda.synchronize()
        for j, r in zip(jobs, ref):
            for got, want in zip(j.outputs(), r):
                assert torch.equal(got.view(torch.uint8), want.view(torch.uint8))
        log("threads rep %d: %d jobs on %d streams bit-identical to serial calls" % (rep, len(jobs), len(jobs)))
