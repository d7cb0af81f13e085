"""Host-side pieces of bench.py: kernel-to-op mapping of profiler names,
algorithmic byte counts, and the one-GPU contract.  No GPU needed."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("name,op", [
    ("resbm::k_enc_fwd_prep", "encode_fwd"),
    ("void resbm::k_enc_fwd<2, 4, 4>(long, int)", "encode_fwd"),
    ("resbm::k_expand<1, 4, false, false, true>", "decode_fwd"),
    ("void resbm::k_expand<2, 4, true, false, false>(long)", "decode_fwd"),
    ("resbm::k_expand<1, 4, false, true, true>", "encode_bwd"),
    ("resbm::k_expand<4, 4, true, true, false>", "encode_bwd"),
    ("_ZN5resbm8k_expandILi1ELi4ELb0ELb1ELb1EEEvliii", "encode_bwd"),
    ("_ZN5resbm8k_expandILi1ELi4ELb0ELb0ELb1EEEvliii", "decode_fwd"),
    ("_ZN5resbm9k_dec_bwdILi2EEEvliiiPKDF16b", "decode_bwd"),
    ("resbm::k_dec_bwd_fin", "decode_bwd"),
    ("_ZN5resbm9k_enc_bwdILi1ELi2ELi4ELi4ELi2EEEvliiii", "encode_bwd"),
    ("resbm::k_rowc_wide<16, 4, false>", "encode_fwd"),
    ("resbm::k_rowc_wide<8, 2, true>", "decode_bwd"),
    ("resbm::k_tokc_wide<16, 4, true, true>", "decode_bwd"),
    ("resbm::k_tokc_wide<8, 2, false, false>", "encode_bwd"),
    ("_ZN5resbm11k_tokc_wideILi8ELi2ELb1ELb1EEEvliii", "decode_bwd"),
    ("_ZN5resbm11k_rowc_wideILi8ELi2ELb0EEEvliii", "encode_fwd"),
    ("resbm::k_expand_wide<8, 2, false, true, true>", "encode_bwd"),
    ("resbm::k_expand_wide<4, 4, true, false, false>", "decode_fwd"),
    ("_ZN5resbm4k_ghEliiPKDF16bPKfPDF16bS4_", "encode_bwd"),
    ("resbm::k_wd_prep", "decode_bwd"),
    ("resbm::k_enc_bwd_fin", "encode_bwd"),
    ("resbm_mx::k_mx_rows<1>", None),
    ("__amd_rocclr_copyBuffer", None),
])
def test_kernel_op(name, op):
    assert bench.kernel_op(name) == op


def test_op_bytes_headline():
    b = bench.op_bytes(16384, 4096, 32)
    assert set(b) == set(bench.OPS)
    # 10 n + 22 r bytes per token plus 24 n r for the weights: 685.8 MB at T = 16384, n = 4096, r = 32
    assert sum(b.values()) == 16384 * (10 * 4096 + 22 * 32) + 24 * 4096 * 32
    assert abs(sum(b.values()) / 1e6 - 685.8) < 0.05


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
