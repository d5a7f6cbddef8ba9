"""bench.py's host-side contract (CPU only): the multi-GPU refusal, the
counter record lookup and the algorithmic byte model of the round."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_counter_record_is_keyed_to_the_kernel():
    with open(bench.TRAFFIC_FILE) as fh:
        rec = json.load(fh)
    assert bench.measured_traffic("gemm.swiglu N=1 K=1 M=1") is None     # another kernel: no record
    t = bench.measured_traffic(rec["kernel"])
    if t is not None:                                                     # the built library's code matches
        assert t == rec["fetch_bytes"] + rec["write_bytes"]
        assert 1.0 <= t / 201850880 < 1.02                               # within 2 % of the algorithmic bytes


class _Dims:
    """The runtime's dimension record, as the byte model reads it."""
    def __init__(self, dtype, d, n_layers, q_dim, kv_dim, ffn, vocab, m, n_draft, d_h):
        self.dtype, self.d, self.n_layers, self.q_dim, self.kv_dim = dtype, d, n_layers, q_dim, kv_dim
        self.ffn, self.vocab, self.m, self.n_draft_layers, self.d_h = ffn, vocab, m, n_draft, d_h


class _Rt:
    def __init__(self, dims, block, qkv_parts=2):
        self.dims, self.block, self._qp = dims, block, qkv_parts

    @property
    def qkv_parts(self):
        return self._qp


def test_gemm_byte_model_at_the_8b_shape():
    """The per-round GEMM bytes at the Qwen3-8B shape, b = 1, B = 16, against
    the weight sizes written out: every weight streamed once per round."""
    dm = _Dims("bf16", 4096, 36, 4096, 1024, 12288, 151936, 5, 5, 4096)
    gb, nl = bench.gemm_bytes(_Rt(dm, 16), 1)
    d, L, Ld, f, V = 4096, 36, 5, 12288, 151936
    qkv, o, gu, dn = d * (d + 2 * 1024), d * d, 2 * f * d, f * d
    weights = (L + Ld) * (qkv + o + gu + dn) * 2 + 2 * V * d * 2 + 5 * d * d * 2 \
        + (3 * d * 4096 + 4096 * 2 * d) * 2 + Ld * 2 * 1024 * d * 2
    assert weights <= gb <= weights * 1.01, (gb, weights)
    assert nl == (L + Ld) * 4 + 2 + 1 + 2 + 1


def test_traffic_record_arithmetic(tmp_path, monkeypatch):
    """The record writer scales each counter's mean per dispatch of the
    dominant kernel by the same counter's reading for the calibration copy
    (synthetic counter files; the digest lookup is stubbed)."""
    import paper_2609_06498_amd.codeobj as co
    name, symbol, pretty, _ = bench.TRAFFIC_KERNEL
    hdr = "Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n"

    def csv_file(path, counter, copy_kib, vals):
        rows = [f'1,"{bench.COPY_KERNEL}",{counter},1.5', f'2,"{bench.COPY_KERNEL}",{counter},{copy_kib}']
        rows += [f'{3 + i},"void dflow::{pretty}(dflow::GemmParams)",{counter},{v}' for i, v in enumerate(vals)]
        rows.append(f'99,"void dflow::other_kernel()",{counter},12345')
        path.write_text(hdr + "\n".join(rows) + "\n")
        return str(path)

    f = csv_file(tmp_path / "f.csv", "FETCH_SIZE", 131072.0, [1000.0, 1002.0])
    w = csv_file(tmp_path / "w.csv", "WRITE_SIZE", 262144.0, [768.0, 768.0])
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    monkeypatch.setattr(co, "kernel_code_digest", lambda lib, sym: "d" * 64)
    bench.write_traffic_record(f, w, copy_mib=256)
    rec = json.loads((tmp_path / "traffic.json").read_text())
    assert rec["kernel"] == name and rec["symbol"] == symbol and rec["code_sha256"] == "d" * 64
    assert rec["fetch_factor"] == 0.5 and rec["write_factor"] == 1.0 and rec["dispatches"] == 2
    assert rec["fetch_bytes"] == 1001 * 1024 * 2 and rec["write_bytes"] == 768 * 1024


def test_profiled_steps_fit_the_event_record():
    """The per-launch event pass never records more launches than the
    library holds (the 32B shape at 64 steps once overflowed it)."""
    import bench
    # 8B shape, b = 1: ~170 GEMM launches and 41 attention launches per round
    assert bench.profiled_steps(128, 1, 170, 41) == 64
    # 32B shape: 64 + 5 layers -> 45 rounds fit
    k = bench.profiled_steps(64, 1, 290, 69)
    assert k * (290 + 69) <= bench.PROF_EVENTS < (k + 1) * (290 + 69)
    # rollouts: rounds per step divide the 64-round target
    assert bench.profiled_steps(10, 3, 3 * 100, 20) == 10
    assert bench.profiled_steps(100, 3, 3 * 100, 20) == 21
    # never zero
    assert bench.profiled_steps(8, 1, 10 ** 6, 10) == 1
