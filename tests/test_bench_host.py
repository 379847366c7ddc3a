"""Host-side pieces of bench.py (no GPU): the counter summaries are only used
while the kernel sources they were taken on are unchanged, and the decode
workloads have the stacked LLaMA shapes they claim."""
import os

import bench


def _summary(tmp_path, kind, hash_value, nbytes):
    p = tmp_path / f"{kind}_w_hbm_traffic.md"
    key = bench.TRAFFIC_KINDS[kind][1]
    p.write_text(f"# x\n\n- HBM bytes per launch: {nbytes:.6e}\n- {key}: `{hash_value}`\n")
    return str(p)


def test_traffic_read_only_on_matching_sources(tmp_path, monkeypatch):
    for kind in bench.TRAFFIC_KINDS:
        good = _summary(tmp_path, kind, bench.source_hash(kind), 1.25e9)
        monkeypatch.setattr(bench, "traffic_file", lambda w, k="gemm_fwd", p=good: p)
        assert bench.read_traffic("w", kind) == 1.25e9
        stale = _summary(tmp_path, kind, "0123456789abcdef", 1.25e9)
        monkeypatch.setattr(bench, "traffic_file", lambda w, k="gemm_fwd", p=stale: p)
        assert bench.read_traffic("w", kind) is None
    monkeypatch.setattr(bench, "traffic_file", lambda w, k="gemm_fwd": str(tmp_path / "none.md"))
    assert bench.read_traffic("w") is None


def test_committed_summaries_name_existing_sources():
    for kind, (sources, _, _, _) in bench.TRAFFIC_KINDS.items():
        for rel in sources:
            assert os.path.exists(os.path.join(bench.ROOT, rel)), rel


def test_decode_shapes():
    assert bench.decode_linears("llama7b") == (("qkv", 12288, 4096), ("o", 4096, 4096),
                                               ("gate_up", 22016, 4096), ("down", 4096, 11008))
    blocks, hid, ffn = bench.DECODE_MODELS["llama65b"]
    assert (blocks, hid, ffn) == (80, 8192, 22016)
    # weights per 7B block: the seven linears' 202,375,168 parameters
    assert sum(c_out * c_in for _, c_out, c_in in bench.decode_linears("llama7b")) == 202375168
