"""Host-side checks of the libchunk C-ABI (no GPU needed):

* the built library loads and exports every function the headers declare
* the canonical parameter layout equals the input recipe's layout
* 1F1B generation and Order validation agree with the Order oracle
  (hand-listed cases, the paper's listing, random permutations)
* descriptor, workspace and argument errors come back as status codes
"""
import ctypes
import os
import re

import numpy as np
import pytest

import synth
from oracle import order as OO
from paper_2606_11169_amd import libchunk as lc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("libchunk.h", "libchunk_ops.h"):
        txt = open(os.path.join(ROOT, "include", h)).read()
        txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(",
                             txt, flags=re.M):
            names.add(m.group(1))
    return sorted(names)


def test_library_exports_every_declared_function():
    L = lc.lib()
    names = declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(lc.EXPORTED)


def desc_of(cfg):
    return lc.desc_of_config(cfg)


TID = {"wq": lc.LC_T_WQ, "wk": lc.LC_T_WK, "wv": lc.LC_T_WV, "wo": lc.LC_T_WO,
       "g1": lc.LC_T_G1, "w1": lc.LC_T_W1, "w3": lc.LC_T_W3, "w2": lc.LC_T_W2,
       "g2": lc.LC_T_G2, "wr": lc.LC_T_WR, "qn": lc.LC_T_QN, "kn": lc.LC_T_KN}


@pytest.mark.parametrize("cfg", list(synth.STAGES.values()), ids=list(synth.STAGES))
def test_param_layout_matches_recipe(cfg):
    d = desc_of(cfg)
    assert lc.lc_param_count(d) == synth.param_count(cfg)
    for name, off, shape in synth.layout(cfg):
        parts = name.split(".")
        layer = int(parts[0][1:])
        expert = int(parts[1][1:]) if len(parts) == 3 else 0
        o, sh = lc.lc_param_offset(d, layer, TID[parts[-1]], expert)
        assert o == off, name
        assert sh == (shape + (1,))[:2], name


def test_param_counts_of_the_workloads():
    assert synth.param_count(synth.TINY_FP32) == 395_776
    assert synth.param_count(synth.LLAMA_2K) == 411_074_560
    assert synth.param_count(synth.STAGE_7B) == 809_533_440
    assert synth.param_count(synth.MOE_2K) == 344_014_848


@pytest.mark.parametrize("M,P,s", [(4, 2, 0), (16, 8, 0), (16, 8, 7), (3, 5, 1), (1, 1, 0),
                                   (8, 4, 2), (5, 8, 0)])
def test_1f1b_matches_oracle(M, P, s):
    got = lc.lc_order_1f1b(M, P, s)
    want = [(mb, lc.LC_PASS_F if ps == "F" else lc.LC_PASS_B) for mb, ps in OO.one_f_one_b(M, P, s)]
    assert got == want


PASS = {"F": lc.LC_PASS_F, "B": lc.LC_PASS_B, "Bi": lc.LC_PASS_BI, "Bw": lc.LC_PASS_BW}


def to_c(entries):
    """Oracle Order -> C entries; a nested pair's first entry carries
    LC_ORDER_WITH_NEXT."""
    out = []
    for e in entries:
        if isinstance(e, list):
            for k, (mb, ps) in enumerate(e):
                out.append((mb, PASS[ps] | (lc.LC_ORDER_WITH_NEXT if k < len(e) - 1 else 0)))
        else:
            out.append((e[0], PASS[e[1]]))
    return out


STATUS = {"OK": lc.LC_OK, "BAD_ORDER": lc.LC_ERR_BAD_ORDER, "STASH_FULL": lc.LC_ERR_STASH_FULL}


def test_validate_matches_oracle_on_fixture_and_random_orders():
    from tests.test_oracle_order import golden_cases
    for M, status, peak, body in golden_cases():
        st, pk = lc.lc_order_validate(to_c(OO.parse(body)), M, M)
        assert st == STATUS[status], body
        if status == "OK":
            assert pk == peak
    rng = np.random.default_rng(0)
    for trial in range(3000):
        M = int(rng.integers(1, 6))
        base = [(i, "F") for i in range(M)] + [(i, "B") for i in range(M)]
        kind = trial % 3
        if kind == 0:
            seq = [base[i] for i in rng.permutation(len(base))]
        elif kind == 1:
            seq = OO.one_f_one_b(M, int(rng.integers(1, 6)), 0)
        else:
            seq = list(base)
            if len(seq) > 1:
                i, j = rng.integers(0, len(seq), size=2)
                seq[i] = seq[j]
        cap = int(rng.integers(1, M + 2))
        st_o, pk_o = OO.validate(seq, M, cap)
        st_c, pk_c = lc.lc_order_validate(to_c(seq), M, cap)
        assert st_c == STATUS[st_o], (seq, cap)
        if st_o == "OK":
            assert pk_c == pk_o


@pytest.mark.parametrize("M,P,s,wd", [(4, 2, 0, 0), (4, 2, 0, 1), (3, 5, 1, 5), (3, 1, 0, 1),
                                      (16, 8, 0, 7), (16, 8, 7, 0), (5, 8, 2, 2), (1, 1, 0, 3)])
def test_1f1b_split_matches_oracle(M, P, s, wd):
    assert lc.lc_order_1f1b_split(M, P, s, wd) == to_c(OO.one_f_one_b_split(M, P, s, wd))


def test_validate_split_matches_oracle_on_rules_and_random_orders():
    from tests.test_oracle_order import SPLIT_RULES
    for M, body, status, peak in SPLIT_RULES:
        st, pk, _ = lc.lc_order_validate_split(to_c(OO.parse(body)), M, M, M)
        assert st == STATUS[status], body
        if status == "OK":
            assert pk == peak
    rng = np.random.default_rng(1)
    names = ["F", "B", "Bi", "Bw"]
    for trial in range(4000):
        M = int(rng.integers(1, 5))
        kind = trial % 4
        if kind == 0:  # a random split choice per microbatch, then shuffled
            base = []
            for i in range(M):
                base += [(i, "F")] + ([(i, "B")] if rng.random() < 0.4 else [(i, "Bi"), (i, "Bw")])
            seq = [base[i] for i in rng.permutation(len(base))]
        elif kind == 1:
            seq = OO.one_f_one_b_split(M, int(rng.integers(1, 6)), 0, int(rng.integers(0, 4)))
        elif kind == 2:  # a valid Order with one entry's pass or mb changed
            seq = OO.one_f_one_b_split(M, int(rng.integers(1, 6)), 0, int(rng.integers(0, 4)))
            i = int(rng.integers(0, len(seq)))
            if rng.random() < 0.5:
                seq[i] = (seq[i][0], names[int(rng.integers(0, 4))])
            else:
                seq[i] = (int(rng.integers(0, M)), seq[i][1])
        else:  # random entries
            n = int(rng.integers(2 * M, 3 * M + 1))
            seq = [(int(rng.integers(0, M)), names[int(rng.integers(0, 4))]) for _ in range(n)]
        cap = int(rng.integers(1, M + 2))
        wcap = int(rng.integers(0, cap + 1))
        st_o, pk_o = OO.validate(seq, M, cap, max_w_pending=wcap)
        st_c, pk_c, _ = lc.lc_order_validate_split(to_c(seq), M, cap, wcap)
        assert st_c == STATUS[st_o], (seq, cap, wcap)
        if st_o == "OK":
            assert pk_c == pk_o
        # the plain validator bounds pending weight passes by the stash only
        st_p, _ = lc.lc_order_validate(to_c(seq), M, cap)
        assert st_p == STATUS[OO.validate(seq, M, cap, max_w_pending=cap)[0]]


@pytest.mark.parametrize("M,P,s", [(4, 2, 0), (16, 8, 0), (3, 5, 1), (2, 2, 0), (5, 1, 0),
                                   (1, 1, 0)])
def test_1f1b_overlap_matches_oracle(M, P, s):
    assert lc.lc_order_1f1b_overlap(M, P, s) == to_c(OO.one_f_one_b_overlap(M, P, s))


@pytest.mark.parametrize("M,P,s,wd", [(8, 4, 0, 1), (8, 4, 0, 0), (16, 8, 0, 2), (3, 5, 1, 1),
                                      (4, 1, 0, 1), (1, 1, 0, 0), (16, 8, 0, 7)])
def test_1f1b_split_overlap_matches_oracle(M, P, s, wd):
    assert lc.lc_order_1f1b_split_overlap(M, P, s, wd) == to_c(
        OO.one_f_one_b_split_overlap(M, P, s, wd))


def test_overlapped_pairs_match_oracle():
    from tests.test_oracle_order import PAIR_RULES
    for M, body, status, peak in PAIR_RULES:
        st, pk = lc.lc_order_validate(to_c(OO.parse(body)), M, M)
        assert st == STATUS[status], body
        if status == "OK":
            assert pk == peak
    # a flagged last entry has no partner
    F, B, NX = lc.LC_PASS_F, lc.LC_PASS_B, lc.LC_ORDER_WITH_NEXT
    assert lc.lc_order_validate([(0, F), (0, B | NX)], 1, 1)[0] == lc.LC_ERR_BAD_ORDER
    assert lc.lc_order_validate([(0, F | 0x200), (0, B)], 1, 1)[0] == lc.LC_ERR_BAD_ORDER
    rng = np.random.default_rng(2)
    names = ["F", "B", "Bi", "Bw"]
    for trial in range(3000):
        M = int(rng.integers(1, 5))
        if trial % 2:
            flat = OO.one_f_one_b_split(M, int(rng.integers(1, 6)), 0, int(rng.integers(0, 4)))
        else:
            flat = OO.one_f_one_b(M, int(rng.integers(1, 6)), 0)
        if trial % 5 == 0 and flat:
            i = int(rng.integers(0, len(flat)))
            flat[i] = (int(rng.integers(0, M)), names[int(rng.integers(0, 4))])
        seq, i = [], 0
        while i < len(flat):  # nest random adjacent pairs, sometimes swapped
            if i + 1 < len(flat) and rng.random() < 0.4:
                pair = [flat[i], flat[i + 1]]
                if rng.random() < 0.5:
                    pair.reverse()
                seq.append(pair)
                i += 2
            else:
                seq.append(flat[i])
                i += 1
        cap = int(rng.integers(1, M + 2))
        wcap = int(rng.integers(0, cap + 1))
        st_o, pk_o = OO.validate(seq, M, cap, max_w_pending=wcap)
        st_c, pk_c, _ = lc.lc_order_validate_split(to_c(seq), M, cap, wcap)
        assert st_c == STATUS[st_o], (seq, cap, wcap)
        if st_o == "OK":
            assert pk_c == pk_o


def test_weight_pass_slots_in_the_workspace():
    d = desc_of(synth.STAGE_7B)
    w0 = lc.lc_workspace_bytes(d, 8)
    w2 = lc.lc_workspace_bytes(d, 8, 2)
    T, D, F, L = 4096, 4096, 11008, 4
    # per layer: dy, dh [T,d], dgate|dup [T,2f], dq|dk|dv [T,3d] (bf16), two
    # norm partial-sum blocks (T/16 rows of d fp32)
    per = L * (2 * (T * D * 2) + T * 2 * F * 2 + T * 3 * D * 2 + 2 * (T // 16) * D * 4)
    assert 2 * per <= w2 - w0 <= 2 * (per + L * 6 * 256)
    with pytest.raises(lc.LibchunkError) as e:
        lc.lc_workspace_bytes(d, 2, 3)
    assert e.value.status == lc.LC_ERR_INVALID_ARG
    # mixture of experts: dy, dh, dq|dk|dv and the norm partials as above,
    # dgate|dup over the 2T routed rows, the routed dy rows [2T, d], the
    # router logit gradients [T, 2] fp32 and the router gradient's partial
    # sums (T/128 blocks x E x d fp32)
    m = desc_of(synth.MOE_2K)
    T, D, FE, E, L = 4096, 2048, 1408, 8, 4
    per = L * (2 * (T * D * 2) + 2 * T * 2 * FE * 2 + T * 3 * D * 2 + 2 * (T // 16) * D * 4
               + 2 * T * D * 2 + T * 2 * 4 + (T // 128) * E * D * 4)
    m0, m1 = lc.lc_workspace_bytes(m, 2, 0), lc.lc_workspace_bytes(m, 2, 1)
    assert per <= m1 - m0 <= per + L * 9 * 256


def test_workspace_grows_with_stash_slots():
    d = desc_of(synth.STAGE_7B)
    w1 = lc.lc_workspace_bytes(d, 1)
    w8 = lc.lc_workspace_bytes(d, 8)
    slot = (w8 - w1) // 7
    T, D, F, L = 4096, 4096, 11008, 4
    # per layer: x, h (fp32 [T,d]); n1, o, n2 (bf16 [T,d]); q, k, v (fp16 [T,d])
    # and their bf16 copy; gate, up (fp32 [T,f]); act (bf16 [T,f]); rstd1,
    # rstd2, lse (fp32 rows)
    approx = L * (4 * T * D * 2 + 2 * T * D * 3 + 2 * T * D * 3 + 2 * T * D * 3 + 4 * T * F * 2
                  + 2 * T * F + 4 * T * (2 + 32))
    assert approx <= slot <= approx + L * 16 * 256


def test_descriptor_errors():
    base = dict(n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ff=512, seq_len=128,
                micro_batch=1, bf16=True)
    assert lc.lc_param_count(lc.make_desc(**base)) > 0
    bad = [dict(d_model=250), dict(n_layers=0), dict(head_dim=64, n_heads=4),
           dict(seq_len=100), dict(d_ff=-1)]
    for kw in bad:
        with pytest.raises(lc.LibchunkError) as e:
            lc.lc_param_count(lc.make_desc(**{**base, **kw}))
        assert e.value.status in (lc.LC_ERR_INVALID_ARG, lc.LC_ERR_UNSUPPORTED)
    with pytest.raises(lc.LibchunkError) as e:
        lc.lc_param_count(lc.make_desc(**base, causal=0))
    assert e.value.status == lc.LC_ERR_UNSUPPORTED
    with pytest.raises(lc.LibchunkError):
        lc.lc_param_offset(lc.make_desc(**base), 1, lc.LC_T_WQ)
    with pytest.raises(lc.LibchunkError):
        lc.lc_param_offset(lc.make_desc(**base), 0, lc.LC_T_WR)


def test_stage_create_argument_errors_before_any_device_work():
    d = lc.make_desc(1, 256, 2, 128, 512, 128, 1, True)
    need = lc.lc_workspace_bytes(d, 2)
    with pytest.raises(lc.LibchunkError) as e:
        lc.lc_stage_create(d, 0, need, 2)
    assert e.value.status == lc.LC_ERR_INVALID_ARG
    with pytest.raises(lc.LibchunkError) as e:
        lc.lc_stage_create(d, 1 << 20, need - 1, 2)
    assert e.value.status == lc.LC_ERR_WORKSPACE
    with pytest.raises(lc.LibchunkError) as e:
        lc.lc_stage_create(d, (1 << 20) + 16, need, 2)
    assert e.value.status == lc.LC_ERR_INVALID_ARG


def test_buffer_entry_points_reject_bad_arguments():
    with pytest.raises(lc.LibchunkError) as e:
        lc.chunk_accumulate_grad(0, 0, lc.LC_FP32, 10)
    assert e.value.status == lc.LC_ERR_INVALID_ARG
    with pytest.raises(lc.LibchunkError):
        lc.chunk_accumulate_grad(4096, 4096 + 16, lc.LC_FP32, 10)  # overlap
    with pytest.raises(lc.LibchunkError):
        lc.chunk_accumulate_grad(4096 + 4, 1 << 20, lc.LC_FP32, 10)  # unaligned
    with pytest.raises(lc.LibchunkError) as e:
        lc.shard_adam_step(4096, 8192, 12288, 16384, lc.LC_BF16, 0, 8, 1e-3, 0.9, 0.999, 1e-8,
                           0.0, 0)
    assert e.value.status == lc.LC_ERR_INVALID_ARG
    assert lc.chunk_accumulate_grad(0, 0, lc.LC_FP32, 0) == lc.LC_OK  # n = 0 is a no-op
    with pytest.raises(lc.LibchunkError):
        lc.lc_gemm(lc.LC_BF16, lc.LC_EPI_STORE, 0, 8, 8, 4096, 8, 1, 4096, 8, 1, 4096, 8)
    with pytest.raises(lc.LibchunkError):
        lc.lc_attention_forward(lc.LC_BF16, lc.LC_BF16, 1, 128, 2, 64, 4096, 4096, 4096, 256,
                                4096, 256, 4096)
    with pytest.raises(lc.LibchunkError):  # fp16 q/k/v need bf16 outputs
        lc.lc_attention_forward(lc.LC_FP16, lc.LC_FP16, 1, 128, 2, 128, 4096, 4096, 4096, 768,
                                4096, 256, 4096)
    with pytest.raises(lc.LibchunkError):  # gemm fp32 operands with a bf16 output
        lc.lc_gemm(lc.LC_FP32, lc.LC_EPI_STORE, 8, 8, 8, 4096, 8, 1, 4096, 8, 1, 4096, 8,
                   c_dtype=lc.LC_BF16)
    with pytest.raises(lc.LibchunkError):  # norm with an unknown dtype
        lc.lc_rmsnorm_forward(4, 8, 4096, 4096, 1e-5, 4096, 4096, 7, lc.LC_BF16, lc.LC_BF16)


def test_timer_entry_points_reject_bad_arguments():
    import ctypes
    L = lc.lib()
    assert L.lc_stage_timer_enable(None, 4) == lc.LC_ERR_INVALID_ARG
    n = ctypes.c_int32(-1)
    assert L.lc_stage_timer_read(None, None, None, 0, ctypes.byref(n)) == lc.LC_ERR_INVALID_ARG
    assert n.value == -1


def test_missing_library_fails_loudly():
    """No fallback: without the built HIP library every entry point raises."""
    import subprocess
    import sys
    code = ("from paper_2606_11169_amd import libchunk as lc\n"
            "lc.LIB_PATH = '/nonexistent/libchunk.so'\n"
            "try:\n"
            "    lc.lc_param_count(lc.desc_of_config(__import__('synth').TINY_FP32))\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=str(__import__('pathlib').Path(__file__).resolve().parents[1]),
                         timeout=120)
    assert "raised:" in out.stdout and "is missing" in out.stdout, out.stdout + out.stderr


def test_runner_refuses_to_run_without_a_gpu():
    import torch
    from paper_2606_11169_amd.runner import require_gpu
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(RuntimeError, match="needs a ROCm GPU"):
        require_gpu()


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU's share: --gpus 2 exits with status 2 and a
    message, before touching a GPU."""
    import pathlib
    import subprocess
    import sys
    root = pathlib.Path(__file__).resolve().parents[1]
    out = subprocess.run([sys.executable, str(root / "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, cwd=str(root), timeout=120)
    assert out.returncode == 2
    assert "--gpus 2 is not supported" in out.stderr


def test_bench_reads_the_committed_counter_summaries():
    """The roofline traffic and matrix-core busy figures parse from profiles/
    (a number while the sources match the recorded hashes, else None)."""
    import importlib.util
    import pathlib
    root = pathlib.Path(__file__).resolve().parents[1]
    spec = importlib.util.spec_from_file_location("bench_mod", root / "bench.py")
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    t = bench.measured_traffic()
    assert t is None or t > 0
    b = bench.measured_mfma_busy()
    assert b is None or (0 < b["value"] < 1 and b["source"] == "profiles/stage7b_mfma_busy.md"
                         and b["csrc_sha256_16"] == bench.csrc_hash())
    assert len(bench.csrc_hash()) == 16 and len(bench.gemm_source_hash()) == 16
