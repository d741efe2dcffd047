"""The algorithmic costs behind the bench's roofline entries, checked against
counts worked out by hand from the workload shapes.  CPU only."""
import bench
from paper_2510_27258_amd import inputs as I


def test_dense_chunk_form_flops_per_token():
    # 2 (C^2 + 2 C d + 2 C dv + 2 d^2 + 4 d dv): the dense chunk form with no
    # triangle discount (C = chunk, d = key width, dv = value width)
    assert bench.reference_flops_per_token(128, 128, 128) == 2 * (16384 + 32768 + 32768 + 32768 + 65536) == 360448
    assert bench.reference_flops_per_token(64, 64, 64) == 2 * (4096 + 8192 + 8192 + 8192 + 16384) == 90112
    assert bench.reference_flops_per_token(64, 32, 32) == 2 * (4096 + 4096 + 4096 + 2048 + 4096) == 36864


def test_headline_output_walk_costs():
    # B2 H32 n16384, d = dv = 128, five segments per head with segment 0 of 36
    # 64-token tiles: the output walk covers every token but segment 0's,
    # reading q, k, v in bf16 (3 x 256 B) and writing an fp32 row (512 B),
    # counted densely at the 64-token tile it walks
    w = I.WORKLOADS["hla2-masked-normalized-bf16-B2H32-n16384-d128-C128"]
    c = bench.kernel_costs(w, 5, 64, 36, 56, two_pass=True)
    tok = 2 * 32 * 16384 - 2 * 32 * 36 * 64
    assert tok == 901120
    assert c["walk"] == ("hbm", tok * 1280, tok * 270336)
    assert bench.reference_flops_per_token(64, 128, 128) == 270336


def test_d64_walk_costs():
    # B4 H16 n4096, d = dv = 64: q, k, v in bf16 (3 x 128 B) and an fp32 row (256 B) per token
    w = I.WORKLOADS["hla2-masked-bf16-B4H16-n4096-d64-C64"]
    c = bench.kernel_costs(w, 8, 64, 8, 8)
    tok = 4 * 16 * 4096
    assert c["walk"] == ("hbm", tok * 640, tok * 90112)


def test_backward_launch_bytes():
    # bytes per token and dimension of each backward launch: the r pass reads
    # q, k, k, v (bf16) and writes r (fp32); the u pass reads v, g (fp32), q
    # and writes u; the first dq term reads g, v, r and writes dq, dv reads
    # r, q, g and writes dv, the paired dk walk reads k, q, u and writes dk;
    # the second dq term reads u, k, k and adds to dq (read and written)
    assert bench.BWD_PASS_BYTES["bwd_ru"] == [(2 + 2 + 2 + 2 + 4) + (2 + 4 + 2 + 4)]
    assert bench.BWD_PASS_BYTES["bwd_dq_dv_dk"] == [(4 + 2 + 4 + 4) + (4 + 2 + 4 + 4) + (2 + 2 + 4 + 4)]
    assert bench.BWD_PASS_BYTES["bwd_dq"] == [4 + 2 + 2 + 8]
