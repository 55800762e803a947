"""The benchmark's byte accounting against the per-token figures fixed by the
sizes (V = 151,936, bf16 logits, fp32 gradients): one read of a 303,872-byte
row, one write of a 607,744-byte gradient row, plus the cache entries."""
import bench
import synth

V = 151936
ROW_BF16 = 2 * V    # 303,872
GRAD_F32 = 4 * V    # 607,744


def test_mc16_one_read_one_write():
    w = synth.MC16
    per_tok = bench.algorithmic_bytes(w, "rkl_mc", 1, 0)
    # ids, teacher and behaviour log-probs: 12 bytes per sample, loss 4 bytes
    assert per_tok == ROW_BF16 + GRAD_F32 + 16 * 12 + 4 == 911_616 + 196
    assert bench.second_read_bytes(w, "rkl_mc", 1) == ROW_BF16
    assert per_tok + ROW_BF16 == 1_215_488 + 196


def test_no_is_ablation_reads_no_behaviour_log_probs():
    w = synth.MC16
    assert (bench.algorithmic_bytes(w, "rkl_mc", 1, 0) -
            bench.algorithmic_bytes(w, "rkl_mc_nois", 1, 0)) == 16 * 4


def test_dense_two_rows():
    w = synth.DENSE
    per_tok = bench.algorithmic_bytes(w, "fkl_dense", 1, 0)
    assert per_tok == 2 * ROW_BF16 + GRAD_F32 + 4 == 1_215_488 + 4
    assert per_tok + bench.second_read_bytes(w, "rkl_dense", 1) == 1_823_232 + 4


def test_top_k_renormalised_reads_only_the_support():
    w = synth.TOPK32
    per_tok = bench.algorithmic_bytes(w, "fkl_topk", 1, 0)
    assert per_tok == 32 * 2 + 32 * 8 + GRAD_F32 + 4
    assert bench.second_read_bytes(w, "fkl_topk", 1) == 0
    # the truncated form has a dense gradient: the whole row is read
    assert bench.algorithmic_bytes(w, "fkl_topk_trunc", 1, 0) == ROW_BF16 + 32 * 8 + GRAD_F32 + 4
    assert bench.second_read_bytes(w, "rkl_topk_trunc", 1) == ROW_BF16


def test_masked_rows_cost_one_zero_write():
    w = synth.MC1_RAGGED
    assert bench.algorithmic_bytes(w, "rkl_mc1", 0, 1) == GRAD_F32 + 4
    assert bench.second_read_bytes(w, "rkl_mc1", 0) == 0
