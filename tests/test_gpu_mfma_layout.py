"""The matrix-core lane layouts the kernels assume, one MFMA at a time, and the streaming-read probe.

rp_selftest_mfma forms the operands of a single MFMA from row-major a and b
in the layouts the attention and prefill kernels use (including the V^T
operand read back from LDS with the transposing read, in P V's key order)
and writes the accumulator back in their output layout. Integer inputs keep
every product and sum exact, so the result must equal the matrix product bit
for bit: a transposed operand, a wrong lane-to-row map or a permuted key
order each give a different matrix.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _bf16(x):
    return torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16)


@pytest.mark.parametrize("shape", ["16x16x32", "16x16x16", "16x16x32_lds_tr"])
@pytest.mark.parametrize("seed", [0, 1])
def test_one_mfma_equals_the_matrix_product(shape, seed):
    import paper_2606_26997_amd as rp
    _, M, N, K = rp.RP_SELFTEST_SHAPES[shape]
    print(f"[case] mfma {shape} seed {seed}", flush=True)
    rng = np.random.default_rng(seed)
    a = rng.integers(-8, 9, size=(M, K))
    b = rng.integers(-8, 9, size=(K, N))
    if seed == 1:
        # distinct entries per position, so that any misplaced operand element changes the product
        a = (np.arange(M * K).reshape(M, K) % 17) - 8
        b = (np.arange(K * N).reshape(K, N) * 7 % 19) - 9
    da, db = _bf16(a).cuda(), _bf16(b).cuda()
    dc = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    rp.selftest_mfma(shape, da, db, dc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(dc.cpu().numpy(), (a @ b).astype(np.float32), err_msg=shape)


@pytest.mark.parametrize("nontemporal", [False, True])
def test_stream_read_reads_every_word_once(nontemporal):
    # The probe folds every 32-bit word it reads into its sink with XOR, so the
    # XOR of the sink equals the XOR of the buffer exactly when every word was
    # read once (or an odd number of times) and nothing else entered; a buffer
    # that is not a multiple of the grid's stride checks the ragged end.
    import paper_2606_26997_amd as rp
    print(f"[case] stream_read nontemporal={nontemporal}", flush=True)
    rng = np.random.default_rng(7)
    words = rng.integers(0, 2 ** 32, size=(3 << 18) + 12, dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32)).cuda()
    sink = torch.zeros(rp.RP_STREAM_READ_SINK_WORDS, dtype=torch.int32, device="cuda")
    rp.stream_read(src, words.nbytes, sink, nontemporal=nontemporal)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(words)
