"""bench.py's measurement helpers, on the host: the algorithmic byte model behind
roofline.achieved, the mirror of the library's launch grouping behind
launches_per_step, and the single-GPU guard."""
import subprocess
import sys

import bench
import swan_inputs as si


def test_attention_bytes_is_the_per_unit_byte_model():
    # 32k x 16: per (sequence, KV head) 32640 pruned tokens x (48 + 48) pairs of
    # (2-byte value, 1-byte index), plus 128 dense buffer tokens of keys and values
    w = si.WORKLOADS["llama2_7b_L32k_b16"]
    want = 16 * 32 * (32640 * 96 * 3 + 2 * 128 * 128 * 2)
    assert bench.attention_bytes(w, [32768] * 16, [48] * 16, [48] * 16, 2) == want
    assert want == 4_846_518_272
    # E4M3 values: one byte per value, keys and values alike
    w8 = si.WORKLOADS["llama2_7b_L32k_b16_e4m3"]
    assert bench.attention_bytes(w8, [32768] * 16, [48] * 16, [48] * 16, 2) == \
        16 * 32 * (32640 * 96 * 2 + 2 * 128 * 128 * 2)
    # keys and values with their own k; a sequence shorter than the buffer has no pages
    w77 = si.WORKLOADS["llama2_7b_L32k_b16_k77_v51"]
    assert bench.attention_bytes(w77, [100] + [32768] * 15, [77] * 16, [51] * 16, 2) == \
        32 * (2 * 100 * 128 * 2) + 15 * 32 * (32640 * 128 * 3 + 2 * 128 * 128 * 2)


def test_attention_launches_mirror_the_grouping():
    ks = [48, 32, 32, 64, 48, 32, 96, 48]
    # k_pad 96 and 64 (two thirds) share a launch, so do 48 and 32
    assert bench.attention_launches(ks, ks) == [(12, False), (6, False)]
    w4 = si.WORKLOADS["llama2_7b_prefill16k_b8"]
    # MHA on fp16 storage: one launch, each sequence at its own k_pad
    assert bench.fused_path(w4)
    assert bench.attention_launches(ks, ks, fused=True) == [(12, False)]
    assert bench.launches_per_step(w4, ks, ks) == 1
    assert bench.attn_kernel_name(w4, ks, ks).startswith("attn_fused_kernel")
    wg = si.WORKLOADS["llama3_8b_gqa_L128k_b4"]
    assert not bench.fused_path(wg)
    assert bench.launches_per_step(wg, ks, ks) == 2
    assert bench.attention_launches([48] * 16, [48] * 16, fused=True) == [(6, True)]
    assert bench.attention_launches([48] * 16, [48] * 16) == [(6, True)]
    assert bench.attention_launches([41, 48], [47, 45]) == [(6, True)]  # one k_pad
    assert bench.attention_launches([77] * 4, [51] * 4) == [(10, False)]
    assert bench.attention_launches(ks, ks, merge_pct=-1) == [(12, True), (8, True), (6, True), (4, True)]


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2", "--steps", "1"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)
