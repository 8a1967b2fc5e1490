"""Host-side accounting the benchmark reports: algorithmic decode bytes per token
and prefill flops, pinned to values worked out by hand from the model shapes
(matrices [out, in], bf16 weights and cache), not recomputed with the library's
own formulas."""

from paper_2608_24204_amd import configs


def test_decode_bytes_per_token_8b():
    # 8B shape: 32 layers, d 4096, 32 query / 8 KV heads x 128, FFN 14336, vocab 128256.
    # Per layer: QKV 6144 x 4096 + O 4096 x 4096 + gate|up 28672 x 4096 + down
    # 4096 x 14336 = 25,165,824 + 16,777,216 + 117,440,512 + 58,720,256
    # = 218,103,808 weights; x 32 layers x 2 B = 13,958,643,712 B.
    # LM head 128256 x 4096 x 2 B = 1,050,673,152 B.
    # Cache read at n positions: n x 32 layers x (K, V) x 1024 x 2 B = n x 131,072 B.
    cfg = configs.CONFIGS["8b"]
    assert cfg.decode_bytes_per_token(0) == 13_958_643_712 + 1_050_673_152
    # the benchmark's mean context: prompt 1024 + (256 + 1) / 2, rounded -> 1152
    assert cfg.decode_bytes_per_token(1152) == 15_009_316_864 + 1152 * 131_072
    tok_s = 8e12 / cfg.decode_bytes_per_token(1152)
    assert round(tok_s, 1) == 527.7
    assert round(0.7 * tok_s, 1) == 369.4


def test_decode_bytes_per_token_1b_tied_head_still_read():
    # 1B shape: 16 layers, d 2048, 32 / 8 heads x 64, FFN 8192, vocab 128256, tied.
    # Per layer: 3072 x 2048 + 2048 x 2048 + 16384 x 2048 + 2048 x 8192
    # = 60,817,408 weights; x 16 x 2 B = 1,946,157,056 B.  The tied LM head is the
    # embedding, read once more per token: 128256 x 2048 x 2 B = 525,336,576 B.
    # Cache: 16 layers x 2 x 512 x 2 B = 32,768 B per position.
    cfg = configs.CONFIGS["1b"]
    assert cfg.decode_bytes_per_token(640) == 1_946_157_056 + 525_336_576 + 640 * 32_768


def test_prefill_flops_8b():
    # projections: 2 x 1024 rows x 218,103,808 weights x 32 layers = 14,293,651,161,088
    # causal attention: 32 layers x 4 x 32 heads x 128 x (1024 x 1025 / 2 pairs)
    #   = 524,288 x 524,800 = 275,146,342,400
    # LM head of the last row: 2 x 128256 x 4096 = 1,050,673,152
    cfg = configs.CONFIGS["8b"]
    assert cfg.prefill_flops() == 14_293_651_161_088 + 275_146_342_400 + 1_050_673_152
