"""The measurement tooling (profile_summary.py) on synthetic rocprofv3
counter CSVs: byte counters scaled by what they read for the three 1 GiB
device copies, the verify GEMM launches of each speculative step found
between its stamp kernels and matched to their roles, the traffic record the
benchmark reads, and the attention instruction mix per 64 MFMAs."""
import csv
import json
import os

import pytest

import profile_summary as ps
import synth

GEMM = "void (anonymous namespace)::gemm_kernel<unsigned short, 4, 3, false>(GemmShape, GemmEpi, int)"
STAMP = "void (anonymous namespace)::stamp_kernel(unsigned long long*)"
COPY = "copyBuffer"


def _write(path, dispatches):
    """dispatches: (kernel name, grid size, duration ns, {counter: value})"""
    os.makedirs(os.path.dirname(path), exist_ok=True)
    rows, t = [], 0
    for did, (name, grid, dur, cnt) in enumerate(dispatches, 1):
        for c, v in cnt.items():
            rows.append({"Dispatch_Id": did, "Kernel_Name": name, "Grid_Size": grid, "Start_Timestamp": t,
                         "End_Timestamp": t + dur, "Counter_Name": c, "Counter_Value": v})
        t += dur + 1000
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def _steps(gemm_counters, other_counters, n_steps=2):
    """Stamp kernels around the draft, the verify GEMMs and the tail, as a
    decode step launches them; then three 1 GiB copies."""
    ds = []
    for _ in range(n_steps):
        ds.append((STAMP, 64, 1000, other_counters(None)))
        ds.append((GEMM.replace("4, 3", "1, 3"), 65536, 5000, other_counters(None)))  # a draft GEMM
        ds.append((STAMP, 64, 1000, other_counters(None)))
        for role in gemm_counters:
            ds.append((GEMM, 65536, 20000, role))
        ds.append((STAMP, 64, 1000, other_counters(None)))
        ds.append((STAMP, 64, 1000, other_counters(None)))
    for _ in range(3):
        ds.append((COPY, 1 << 20, 200000, other_counters("copy")))
    return ds


def test_gemm_counters_scaled_by_copies_and_matched_to_roles(tmp_path, monkeypatch):
    monkeypatch.setattr(ps, "OUT_DIR", str(tmp_path))
    wl = synth.WORKLOADS["llama7b_p512"]
    M = len(synth.TREES[wl.tree]) + 1
    roles = ps.verify_roles(wl.model, M)
    # FETCH_SIZE reads half the bytes (KiB) on the copies: factor 2; each GEMM
    # fetches exactly its algorithmic bytes once scaled, and writes 1 MiB
    fetch = [{"FETCH_SIZE": b / 1024 / 2} for _, _, _, b in roles]
    write = [{"WRITE_SIZE": 1024.0} for _ in roles]
    sq = [{"SQ_INSTS_VALU_MFMA_MOPS_BF16": 1e6, "SQ_VALU_MFMA_BUSY_CYCLES": 8e5, "SQ_BUSY_CYCLES": 1e6,
           "GRBM_GUI_ACTIVE": 8e4} for _ in roles]
    d = tmp_path / "pmc"
    _write(str(d / "fetch" / "run_counter_collection.csv"),
           _steps(fetch, lambda k: {"FETCH_SIZE": 524288.0 if k == "copy" else 0.0}))
    _write(str(d / "write" / "run_counter_collection.csv"),
           _steps(write, lambda k: {"WRITE_SIZE": 1048576.0 if k == "copy" else 0.0}))
    _write(str(d / "sq" / "run_counter_collection.csv"),
           _steps(sq, lambda k: {c: 1.0 for c in sq[0]}))
    ps.counters(str(d), "llama7b_p512", "F", "W", "S")
    md = (tmp_path / "counters_llama7b_p512.md").read_text()
    assert "factors 2.0000 (fetch) and 1.0000 (write)" in md
    rec = json.loads((tmp_path / "verify_gemm_llama7b_p512_traffic.json").read_text())
    alg = sum(b for *_, b in roles) / len(roles)
    assert rec["fetch_bytes_per_launch"] == pytest.approx(alg)
    assert rec["write_bytes_per_launch"] == pytest.approx(1024 * 1024)
    assert rec["sources_sha256"] == ps.sources_sha()
    # one table row per role: QKV's traffic over algorithmic bytes is
    # (alg + 1 MiB) / alg
    qkv = next(b for r, _, _, b in roles if r == "QKV")
    row = next(line for line in md.splitlines() if line.startswith("| QKV |"))
    assert f"{(qkv + 1048576) / qkv:.3f}" in row
    assert row.split("|")[3].strip() == str(2 * wl.model.n_layers)  # two steps, one QKV per layer


def test_gemm_counters_refuse_a_layer_count_mismatch(tmp_path, monkeypatch):
    monkeypatch.setattr(ps, "OUT_DIR", str(tmp_path))
    wl = synth.WORKLOADS["llama7b_p512"]
    roles = ps.verify_roles(wl.model, 65)[:-1]  # one launch short
    d = tmp_path / "pmc"
    for sub, c, v in (("fetch", "FETCH_SIZE", 524288.0), ("write", "WRITE_SIZE", 1048576.0), ("sq", "GRBM_GUI_ACTIVE", 1.0)):
        _write(str(d / sub / "run_counter_collection.csv"),
               _steps([{c: 1.0} for _ in roles], lambda k, c=c, v=v: {c: v if k == "copy" else 0.0}))
    with pytest.raises(SystemExit):
        ps.counters(str(d), "llama7b_p512", "F", "W", "S")


def test_attention_mix_per_64_mfma(tmp_path, monkeypatch):
    monkeypatch.setattr(ps, "OUT_DIR", str(tmp_path))
    shared = "void (anonymous namespace)::tree_attn_shared<unsigned short, 128>(TreeAttnArgs)"
    window = "void (anonymous namespace)::tree_attn_window<unsigned short, 128>(TreeAttnArgs)"
    base = {"SQ_WAVES": 512.0, "SQ_WAVE_CYCLES": 1.0, "SQ_BUSY_CYCLES": 1.0, "SQ_INSTS_VALU": 512 * 300.0,
            "SQ_INSTS_MFMA": 1024 * 64.0, "SQ_INSTS_LDS": 1024 * 60.0, "SQ_INSTS_SALU": 512 * 10.0,
            "SQ_LDS_BANK_CONFLICT": 1024 * 6.0, "GRBM_GUI_ACTIVE": 1.0}
    ds = []
    for _ in range(2):
        ds += [(STAMP, 64, 1000, base), (STAMP, 64, 1000, base), (shared, 256, 10000, base),
               (window, 256, 6000, dict(base, SQ_INSTS_MFMA=0.0)), (STAMP, 64, 1000, base), (STAMP, 64, 1000, base)]
    _write(str(tmp_path / "sq" / "run_counter_collection.csv"), ds)
    copies = [(COPY, 1 << 20, 200000, {})] * 3
    fetch = [(n, g, t, {"FETCH_SIZE": 524288.0 if n == COPY else (2048.0 if "attn" in n else 0.0)})
             for n, g, t, _ in ds + copies]
    write = [(n, g, t, {"WRITE_SIZE": 1048576.0 if n == COPY else (512.0 if "attn" in n else 0.0)})
             for n, g, t, _ in ds + copies]
    _write(str(tmp_path / "fetch" / "run_counter_collection.csv"), fetch)
    _write(str(tmp_path / "write" / "run_counter_collection.csv"), write)
    ps.attn(str(tmp_path), "llama7b_p512", "CMD", "F", "W")
    md = (tmp_path / "attn_counters_llama7b_p512.md").read_text()
    row = next(line for line in md.splitlines() if line.startswith("| `tree_attn_shared`"))
    cells = [c.strip() for c in row.split("|")[1:-1]]
    # dispatches, dur, waves, VALU/wave, MFMA/wave, LDS/wave, SALU/wave, VALU/64 MFMA, LDS/64 MFMA, conflicts
    assert cells[1] == "2" and cells[2] == "10.00" and cells[3] == "512"
    assert cells[4] == "300.0" and cells[5] == "128.0"
    assert cells[8] == "150" and cells[9] == "60.0" and cells[10] == "0.100"
    wrow = next(line for line in md.splitlines() if line.startswith("| `tree_attn_window`"))
    assert wrow.split("|")[9].strip() == "–"
    # bytes: 2048 KiB fetched x 2 (the copies' factor) = 4.19 MB, 512 KiB written = 0.52 MB
    brow = [line for line in md.splitlines() if line.startswith("| `tree_attn_shared`")][1]
    assert [c.strip() for c in brow.split("|")[3:5]] == ["4.19", "0.52"]
