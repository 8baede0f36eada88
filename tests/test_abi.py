"""C-ABI checks that need no GPU: exported symbols and synchronous argument validation.

Every call here fails validation before anything reaches the HIP runtime.
"""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2606_26997_amd as rp
from paper_2606_26997_amd import _binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "rp.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rp_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 10
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (rp_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    assert set(names) == set(B.EXPORTED)
    lib = rp.load()
    for n in names:
        assert getattr(lib, n) is not None


def test_status_strings():
    for code, tag in [(0, "RP_OK"), (1, "INVALID_ARG"), (2, "UNSUPPORTED"), (3, "WORKSPACE"),
                      (4, "HIP"), (5, "LAYOUT")]:
        assert tag in rp.status_string(code)
    assert "unknown" in rp.status_string(99)


# Fake but 256-aligned "device" addresses: validation never dereferences them.
A = 0x10000000


def _kv(**kw):
    d = dict(k_pages=A, v_pages=A + 4096, k_scale=None, v_scale=None, num_pages=4, num_kv_heads=2,
             page_size=16, head_dim=64, kv_dtype=rp.RP_KV_BF16)
    d.update(kw)
    return B.RpPagedKV(d["k_pages"], d["v_pages"], d["k_scale"], d["v_scale"], d["num_pages"],
                       d["num_kv_heads"], d["page_size"], d["head_dim"], d["kv_dtype"])


def _layout(**kw):
    d = dict(num_seqs=2, num_groups=1, num_q_heads=4, seq_to_group=A, prefix_lens=A, pbt=A, mpp=2,
             resp_lens=A, rbt=A, mrp=2)
    d.update(kw)
    return B.RpGroupLayout(d["num_seqs"], d["num_groups"], d["num_q_heads"], d["seq_to_group"],
                           d["prefix_lens"], d["pbt"], d["mpp"], d["resp_lens"], d["rbt"], d["mrp"])


def _ws_size(kv, layout):
    n = ctypes.c_size_t(0)
    st = rp.load().rp_group_decode_attn_workspace_size(ctypes.byref(kv) if kv is not None else None,
                                                       ctypes.byref(layout) if layout is not None else None,
                                                       ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("kv_kw,lay_kw,status,needle", [
    (dict(k_pages=None), {}, rp.RP_ERR_INVALID_ARG, "NULL"),
    (dict(k_pages=A + 8), {}, rp.RP_ERR_INVALID_ARG, "aligned"),
    (dict(page_size=32), {}, rp.RP_ERR_UNSUPPORTED, "page_size"),
    (dict(head_dim=96), {}, rp.RP_ERR_UNSUPPORTED, "head_dim"),
    (dict(kv_dtype=rp.RP_KV_FP8_E4M3), {}, rp.RP_ERR_INVALID_ARG, "scale"),
    (dict(k_scale=A), {}, rp.RP_ERR_INVALID_ARG, "NULL for bf16"),
    (dict(kv_dtype=7), {}, rp.RP_ERR_UNSUPPORTED, "kv_dtype"),
    (dict(num_pages=0), {}, rp.RP_ERR_INVALID_ARG, "num_pages"),
    ({}, dict(num_q_heads=3), rp.RP_ERR_INVALID_ARG, "multiple"),
    ({}, dict(num_q_heads=6), rp.RP_ERR_UNSUPPORTED, "ratio"),
    ({}, dict(num_groups=0), rp.RP_ERR_INVALID_ARG, "num_groups"),
    ({}, dict(seq_to_group=None), rp.RP_ERR_INVALID_ARG, "NULL"),
    ({}, dict(rbt=None), rp.RP_ERR_INVALID_ARG, "resp_block_table"),
    ({}, dict(num_seqs=-1), rp.RP_ERR_INVALID_ARG, "num_seqs"),
])
def test_invalid_arguments_rejected(kv_kw, lay_kw, status, needle):
    st, _ = _ws_size(_kv(**kv_kw), _layout(**lay_kw))
    assert st == status
    assert needle in rp.last_error()


def test_planner_group_limit():
    # 4096 groups is the largest plan; one more is refused before any launch.
    assert _ws_size(_kv(), _layout(num_groups=4096))[0] == rp.RP_OK
    st, _ = _ws_size(_kv(), _layout(num_groups=4097))
    assert st == rp.RP_ERR_UNSUPPORTED and "limit" in rp.last_error()


def test_null_structs_rejected():
    assert _ws_size(None, _layout())[0] == rp.RP_ERR_INVALID_ARG
    assert _ws_size(_kv(), None)[0] == rp.RP_ERR_INVALID_ARG


def test_workspace_size_depends_only_on_scalars_and_grows():
    st, n1 = _ws_size(_kv(), _layout(mrp=2))
    st2, n2 = _ws_size(_kv(), _layout(mrp=200))
    assert st == st2 == rp.RP_OK and 0 < n1 < n2
    assert _ws_size(_kv(), _layout(num_seqs=0))[1] == 0


def test_short_or_misaligned_workspace_rejected():
    kv, lay = _kv(), _layout()
    _, need = _ws_size(kv, lay)
    lib = rp.load()
    st = lib.rp_plan(ctypes.byref(kv), ctypes.byref(lay), A, need - 1, None)
    assert st == rp.RP_ERR_WORKSPACE and "needs" in rp.last_error()
    st = lib.rp_plan(ctypes.byref(kv), ctypes.byref(lay), A + 64, need, None)
    assert st == rp.RP_ERR_WORKSPACE and "aligned" in rp.last_error()
    st = lib.rp_group_decode_attn(ctypes.byref(kv), ctypes.byref(lay), A, ctypes.c_float(0.1), A, None,
                                  None, need, None)
    assert st == rp.RP_ERR_WORKSPACE


def test_attention_and_append_pointer_checks():
    kv, lay = _kv(), _layout()
    _, need = _ws_size(kv, lay)
    lib = rp.load()
    st = lib.rp_group_decode_attn(ctypes.byref(kv), ctypes.byref(lay), None, ctypes.c_float(0.1), A, None,
                                  A, need, None)
    assert st == rp.RP_ERR_INVALID_ARG and "q" in rp.last_error()
    st = lib.rp_group_decode_attn(ctypes.byref(kv), ctypes.byref(lay), A, ctypes.c_float(0.1), A + 2, None,
                                  A, need, None)
    assert st == rp.RP_ERR_INVALID_ARG and "out" in rp.last_error()
    assert lib.rp_kv_append(ctypes.byref(kv), ctypes.byref(lay), None, A, None) == rp.RP_ERR_INVALID_ARG
    assert lib.rp_kv_append(ctypes.byref(kv), ctypes.byref(_layout(mrp=0)), A, A, None) == rp.RP_ERR_INVALID_ARG


def test_lse_combine_argument_checks():
    lib = rp.load()
    assert lib.rp_lse_combine(A, A, A, 4, 96, A, None, None) == rp.RP_ERR_UNSUPPORTED
    assert lib.rp_lse_combine(A, A, None, 4, 128, A, None, None) == rp.RP_ERR_INVALID_ARG
    assert lib.rp_lse_combine(A, A, A, -1, 128, A, None, None) == rp.RP_ERR_INVALID_ARG
    assert lib.rp_lse_combine(None, None, None, 0, 128, None, None, None) == rp.RP_OK


def test_empty_batch_is_a_no_op():
    kv, lay = _kv(), _layout(num_seqs=0)
    lib = rp.load()
    assert lib.rp_group_decode_attn(ctypes.byref(kv), ctypes.byref(lay), None, ctypes.c_float(0.1), None,
                                    None, None, 0, None) == rp.RP_OK
    assert lib.rp_kv_append(ctypes.byref(kv), ctypes.byref(lay), None, None, None) == rp.RP_OK


def test_binding_raises_with_detail():
    with pytest.raises(rp.RpError) as e:
        B._check(rp.RP_ERR_UNSUPPORTED, "x")
    assert e.value.status == rp.RP_ERR_UNSUPPORTED


def test_plan_layout_sections_fit_the_workspace():
    kv, lay = _kv(), _layout(num_seqs=5, num_groups=2, mpp=3, mrp=70)
    _, need = _ws_size(kv, lay)
    info = B.plan_layout(kv, lay)
    offs = [info.hdr, info.grp_off, info.grp_members, info.prefix_items, info.resp_items,
            info.seq_parts, info.part_o, info.part_lse]
    assert offs == sorted(offs) and len(set(offs)) == len(offs)
    assert all(o % 256 == 0 for o in offs)
    # Capacities: 16-page prefix chunks; response pieces of 16 pages, the shortest B, since this
    # layout's response capacity (5 sequences x 70 pages x 2 kv-heads) is at most 2^17 page-heads.
    assert info.max_prefix_items == 2 * 1
    assert info.max_resp_items == 5 * 5
    assert info.parts_per_row == 1 + 5
    assert info.max_parts == 5 * 4 * 6
    assert info.part_lse + 4 * info.max_parts <= need
    assert info.part_o + 4 * info.max_parts * 64 <= info.part_lse
    # Above 2^17 page-heads the slots are sized for 32-page pieces.
    big = B.plan_layout(kv, _layout(num_seqs=1000, num_groups=2, mpp=3, mrp=70))
    assert big.max_resp_items == 1000 * 3 and big.parts_per_row == 1 + 3
    with pytest.raises(B.RpError):
        B.plan_layout(_kv(head_dim=96), lay)


def _prefill_layout(**kw):
    d = dict(num_groups=2, num_q_heads=4, num_tokens=10, offs=A, pbt=A, mpp=2)
    d.update(kw)
    return B.RpPrefillLayout(d["num_groups"], d["num_q_heads"], d["num_tokens"], d["offs"], d["pbt"], d["mpp"])


@pytest.mark.parametrize("lay_kw,status,needle", [
    # One prompt's rows are addressed with 32-bit byte offsets: 2^20 pages x 16 tokens x 2 kv-heads x 64
    # x 2 B = 2^32 bytes is one too many.
    (dict(mpp=1 << 20), rp.RP_ERR_UNSUPPORTED, "too large"),
    (dict(num_q_heads=3), rp.RP_ERR_INVALID_ARG, "multiple"),
    (dict(num_q_heads=6), rp.RP_ERR_UNSUPPORTED, "ratio"),
    (dict(offs=None), rp.RP_ERR_INVALID_ARG, "prompt_offs"),
    (dict(mpp=0), rp.RP_ERR_INVALID_ARG, "max_prefix_pages"),
    (dict(num_tokens=-1), rp.RP_ERR_INVALID_ARG, "num_tokens"),
])
def test_prefill_layout_checks(lay_kw, status, needle):
    lib = rp.load()
    st = lib.rp_prefill_kv_write(ctypes.byref(_kv()), ctypes.byref(_prefill_layout(**lay_kw)), A, A, None)
    assert st == status and needle in rp.last_error()


def test_prefill_pointer_checks():
    lib = rp.load()
    kv, lay = _kv(), _prefill_layout()
    assert lib.rp_prefill_kv_write(ctypes.byref(kv), ctypes.byref(lay), None, A, None) == rp.RP_ERR_INVALID_ARG
    assert lib.rp_prefill_kv_write(ctypes.byref(kv), ctypes.byref(lay), A + 2, A, None) == rp.RP_ERR_INVALID_ARG
    st = lib.rp_prefill_attn(ctypes.byref(kv), ctypes.byref(lay), A, A, A, ctypes.c_float(0.1), None, None, None)
    assert st == rp.RP_ERR_INVALID_ARG and "out" in rp.last_error()
    st = lib.rp_prefill_attn(ctypes.byref(kv), ctypes.byref(lay), A, A, A, ctypes.c_float(0.1), A, A + 2, None)
    assert st == rp.RP_ERR_INVALID_ARG and "lse" in rp.last_error()
    for bad in (0.0, -0.1, float("inf"), float("nan")):
        st = lib.rp_prefill_attn(ctypes.byref(kv), ctypes.byref(lay), A, A, A, ctypes.c_float(bad), A, None, None)
        assert st == rp.RP_ERR_INVALID_ARG and "softmax_scale" in rp.last_error()
    # Nothing to do: returns before touching any pointer.
    assert lib.rp_prefill_attn(ctypes.byref(kv), ctypes.byref(_prefill_layout(num_tokens=0)), None, None, None,
                               ctypes.c_float(0.1), None, None, None) == rp.RP_OK


def test_decode_qk_prep_argument_checks():
    kv, lay = _kv(), _layout()
    lib = rp.load()
    call = lambda kv_, lay_, q=A, k=A, v=A, wq=A, wk=A, eps=1e-6, theta=1e6, qo=A, ko=None: \
        lib.rp_decode_qk_prep(ctypes.byref(kv_), ctypes.byref(lay_), q, k, v, wq, wk, eps, theta, qo, ko, None)
    assert call(kv, lay, q=None) == rp.RP_ERR_INVALID_ARG and "q_in" in rp.last_error()
    assert call(kv, lay, wk=None) == rp.RP_ERR_INVALID_ARG
    assert call(kv, lay, qo=A + 1) == rp.RP_ERR_INVALID_ARG
    assert call(kv, lay, ko=A + 1) == rp.RP_ERR_INVALID_ARG and "k_out" in rp.last_error()
    assert call(kv, lay, eps=-1.0) == rp.RP_ERR_INVALID_ARG and "rms_eps" in rp.last_error()
    assert call(kv, lay, eps=float("nan")) == rp.RP_ERR_INVALID_ARG
    assert call(kv, lay, theta=0.0) == rp.RP_ERR_INVALID_ARG and "rope_theta" in rp.last_error()
    assert call(kv, lay, theta=float("inf")) == rp.RP_ERR_INVALID_ARG
    assert call(kv, _layout(mrp=0)) == rp.RP_ERR_INVALID_ARG and "max_resp_pages" in rp.last_error()
    assert call(_kv(head_dim=96), lay) == rp.RP_ERR_UNSUPPORTED
    # An empty batch launches nothing and needs no pointers.
    assert call(kv, _layout(num_seqs=0), q=None, k=None, v=None, wq=None, wk=None, qo=None) == rp.RP_OK


def test_grpo_advantage_argument_checks():
    lib = rp.load()
    call = lambda r=A, R=4, K=8, eps=1e-6, ddof=1, adv=A, mu=None, sd=None: \
        lib.rp_grpo_advantage(r, R, K, eps, ddof, adv, mu, sd, None)
    assert call(r=None) == rp.RP_ERR_INVALID_ARG and "rewards" in rp.last_error()
    assert call(adv=A + 2) == rp.RP_ERR_INVALID_ARG
    assert call(mu=A + 1) == rp.RP_ERR_INVALID_ARG and "group_mean" in rp.last_error()
    assert call(K=0) == rp.RP_ERR_INVALID_ARG
    assert call(R=-1) == rp.RP_ERR_INVALID_ARG
    assert call(ddof=2) == rp.RP_ERR_INVALID_ARG and "ddof" in rp.last_error()
    assert call(eps=-1e-6) == rp.RP_ERR_INVALID_ARG and "eps_std" in rp.last_error()
    assert call(eps=float("inf")) == rp.RP_ERR_INVALID_ARG
    assert call(R=0, r=None, adv=None) == rp.RP_OK


def test_selftest_mfma_argument_checks():
    lib = rp.load()
    call = lambda shape=0, a=A, b=A, c=A: lib.rp_selftest_mfma(shape, a, b, c, None)
    assert call(shape=3) == rp.RP_ERR_UNSUPPORTED and "shape" in rp.last_error()
    assert call(shape=-1) == rp.RP_ERR_UNSUPPORTED
    assert call(a=None) == rp.RP_ERR_INVALID_ARG and "NULL" in rp.last_error()
    assert call(c=A + 2) == rp.RP_ERR_INVALID_ARG and "aligned" in rp.last_error()
    assert call(b=A + 1) == rp.RP_ERR_INVALID_ARG
    assert sorted(code for code, *_ in rp.RP_SELFTEST_SHAPES.values()) == [0, 1, 2]


def test_stream_read_argument_checks():
    lib = rp.load()
    call = lambda src=A, n=1 << 20, sink=A, nt=0: lib.rp_stream_read(src, n, sink, nt, None)
    assert call(src=None) == rp.RP_ERR_INVALID_ARG and "NULL" in rp.last_error()
    assert call(src=A + 8) == rp.RP_ERR_INVALID_ARG and "aligned" in rp.last_error()
    assert call(sink=A + 2) == rp.RP_ERR_INVALID_ARG
    assert call(n=0) == rp.RP_ERR_INVALID_ARG and "multiple of 16" in rp.last_error()
    assert call(n=24) == rp.RP_ERR_INVALID_ARG


def _no_gpu():
    import torch
    return not torch.cuda.is_available()


@pytest.mark.skipif(not _no_gpu(), reason="forces a HIP runtime failure; only meaningful without a GPU")
def test_hip_failure_maps_to_rp_err_hip():
    """Well-formed calls on a host without a GPU: the first HIP runtime call fails, and the library
    reports RP_ERR_HIP with the runtime's text instead of crashing. rp_plan fails in its device
    query, rp_kv_append and rp_lse_combine in their kernel launches."""
    lib = rp.load()
    kv, lay = _kv(), _layout()
    st, n = _ws_size(kv, lay)
    assert st == rp.RP_OK and n > 0
    st = lib.rp_plan(ctypes.byref(kv), ctypes.byref(lay), A, n, None)
    assert st == rp.RP_ERR_HIP, rp.status_string(st)
    assert "hipGetDevice" in rp.last_error()
    st = lib.rp_kv_append(ctypes.byref(kv), ctypes.byref(lay), A, A, None)
    assert st == rp.RP_ERR_HIP and "append kernel launch" in rp.last_error(), rp.last_error()
    st = lib.rp_lse_combine(A, A, A, 4, 64, A, None, None)
    assert st == rp.RP_ERR_HIP and "combine kernel launch" in rp.last_error(), rp.last_error()
    # The binding turns the code into an exception carrying the same detail.
    with pytest.raises(rp.RpError) as e:
        B._check(lib.rp_plan(ctypes.byref(kv), ctypes.byref(lay), A, n, None), "rp_plan")
    assert e.value.status == rp.RP_ERR_HIP and "hipGetDevice" in str(e.value)


def test_noalloc_scratch_limit_and_refusal():
    """The binding's scratch size is the header's, and a layout whose workspace exceeds it is refused
    before anything reaches the HIP runtime."""
    text = open(HEADER).read()
    m = re.search(r"#define RP_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == rp.RP_NOALLOC_SCRATCH_BYTES
    kv = _kv(num_kv_heads=8, head_dim=128)
    lay = _layout(num_seqs=1024, num_groups=64, num_q_heads=16, mpp=16, mrp=513)
    st, need = _ws_size(kv, lay)
    assert st == rp.RP_OK and need > rp.RP_NOALLOC_SCRATCH_BYTES
    lib = rp.load()
    st = lib.rp_group_decode_attn_noalloc(ctypes.byref(kv), ctypes.byref(lay), A, ctypes.c_float(0.1), A, None,
                                          None)
    assert st == rp.RP_ERR_WORKSPACE and "static scratch" in rp.last_error()
    assert lib.rp_group_decode_attn_noalloc(ctypes.byref(kv), ctypes.byref(_layout(num_seqs=0, num_q_heads=16)), None,
                                            ctypes.c_float(0.1), None, None, None) == rp.RP_OK
    assert lib.rp_group_decode_attn_noalloc(ctypes.byref(_kv(head_dim=96)), ctypes.byref(lay), A,
                                            ctypes.c_float(0.1), A, None, None) == rp.RP_ERR_UNSUPPORTED


def test_decode_qk_prep_plan_argument_checks():
    """The fused prep + plan call checks the prep's arguments and the plan's workspace before any launch."""
    kv, lay = _kv(), _layout()
    lib = rp.load()
    _, need = _ws_size(kv, lay)
    call = lambda lay_=lay, q=A, eps=1e-6, ws=A, n=need: lib.rp_decode_qk_prep_plan(
        ctypes.byref(kv), ctypes.byref(lay_), q, A, A, A, A, eps, 1e6, A, None, ws, n, None)
    assert call(q=None) == rp.RP_ERR_INVALID_ARG and "q_in" in rp.last_error()
    assert call(eps=-1.0) == rp.RP_ERR_INVALID_ARG and "rms_eps" in rp.last_error()
    assert call(n=need - 1) == rp.RP_ERR_WORKSPACE
    assert call(ws=A + 64) == rp.RP_ERR_WORKSPACE
    assert call(ws=None) == rp.RP_ERR_WORKSPACE
    assert call(lay_=_layout(mrp=0), n=_ws_size(kv, _layout(mrp=0))[1]) == rp.RP_ERR_INVALID_ARG
    assert call(lay_=_layout(num_seqs=0), q=None, ws=None, n=0) == rp.RP_OK
