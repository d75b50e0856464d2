"""CPU-only checks of the Python binding's argument checks: every tensor is
checked against the element type the C ABI declares and against the element
count the call's shape arguments imply, before any pointer reaches the
library (a wrong dtype or a short buffer would otherwise be read or written
past its end on the device). Host tensors are used: a correctly typed and
sized argument list gets past every check and stops at the device check."""
import pytest
import torch

import paper_2607_27090_amd as isl

i32, i64, f32, bf16, f64 = torch.int32, torch.int64, torch.float32, torch.bfloat16, torch.float64


def T(n, dt):
    return torch.zeros(max(n, 1), dtype=dt)


def retrieve_args(nq=2, n=100, d=16, k=5, stride=0):
    return dict(query_emb=T(nq * d, f32), bank=T(n * d if stride == 0 else (nq - 1) * stride
                                                 + n * d, f32),
                n=n, d=d, k=k, out_ids=T(nq * k, i32), out_scores=T(nq * k, f32), nq=nq,
                bank_stride=stride, workspace=T(1 << 16, torch.uint8), stream=0)


def call_retrieve(a):
    a = dict(a)
    isl.is_retrieve(a.pop("query_emb"), a.pop("bank"), a.pop("n"), a.pop("d"), a.pop("k"),
                    a.pop("out_ids"), a.pop("out_scores"), **a)


def test_retrieve_well_formed_reaches_the_device_check():
    with pytest.raises(ValueError, match="device tensors"):
        call_retrieve(retrieve_args())
    with pytest.raises(ValueError, match="device tensors"):
        call_retrieve(retrieve_args(stride=100 * 16))


@pytest.mark.parametrize("name,bad,msg", [
    ("out_ids", T(10, i64), "out_ids must be torch.int32"),
    ("out_ids", T(9, i32), "out_ids holds 9 elements"),
    ("out_scores", T(10, torch.float16), "out_scores must be torch.float32"),
    ("out_scores", T(3, f32), "out_scores holds 3"),
    ("bank", T(100 * 16, bf16), "bank must be torch.float32"),
    ("bank", T(99 * 16, f32), "bank holds"),
    ("query_emb", T(31, f32), "query_emb holds 31"),
])
def test_retrieve_rejects_wrong_dtype_or_size(name, bad, msg):
    a = retrieve_args()
    a[name] = bad
    with pytest.raises(ValueError, match=msg):
        call_retrieve(a)


def test_retrieve_per_request_banks_need_the_strided_span():
    a = retrieve_args(stride=100 * 16)
    a["bank"] = T(100 * 16 * 2 - 1, f32)
    with pytest.raises(ValueError, match="bank holds"):
        call_retrieve(a)


def slot_map_args(nq=2, k=4, n=50, mb=9, mt=40, lens_stride=0):
    return dict(ids=T(nq * k, i32), fact_lens=T(n if lens_stride == 0 else
                                                (nq - 1) * lens_stride + n, i32),
                start_pos=3, block_table=T(nq * mb, i32), page_size=16,
                out_slots=T(nq * mt, i64), out_positions=T(nq * mt, i32), out_m=T(nq, i32),
                k=k, nq=nq, n=n, lens_stride=lens_stride, max_blocks=mb, max_tokens=mt,
                status=T(1, i32), stream=0)


def call_slot_map(a):
    a = dict(a)
    isl.is_slot_map(a.pop("ids"), a.pop("fact_lens"), a.pop("start_pos"), a.pop("block_table"),
                    a.pop("page_size"), a.pop("out_slots"), a.pop("out_positions"),
                    a.pop("out_m"), **a)


@pytest.mark.parametrize("name,bad,msg", [
    (None, None, "device tensors"),
    ("out_slots", T(80, i32), "out_slots must be torch.int64"),
    ("out_slots", T(79, i64), "out_slots holds 79"),
    ("out_positions", T(80, i64), "out_positions must be torch.int32"),
    ("ids", T(8, i64), "ids must be torch.int32"),
    ("block_table", T(17, i32), "block_table holds 17"),
    ("fact_lens", T(49, i32), "fact_lens holds 49"),
    ("out_m", T(1, i32), "out_m holds 1"),
    ("status", T(1, i64), "status must be"),
])
def test_slot_map_checks(name, bad, msg):
    a = slot_map_args()
    if name:
        a[name] = bad
    with pytest.raises(ValueError, match=msg):
        call_slot_map(a)


def inject_kw(nq=2, k=4, n=50, mt=40, L=2, H=2, D=16, Ts=300, ns=128):
    return dict(ids=T(nq * k, i32), preK=T(L * Ts * H * D, bf16), V=T(L * Ts * H * D, bf16),
                slots=T(nq * mt, i64), positions=T(nq * mt, i32), paged_k=T(L * ns * H * D, bf16),
                paged_v=T(L * ns * H * D, bf16), fact_offsets=T(n, i64), fact_lens=T(n, i32),
                m=T(nq, i32), k=k, nq=nq, n=n, lens_stride=0, max_tokens=mt, L=L, H=H, D=D,
                T_store=Ts, num_slots=ns, stream=0)


def call_inject(a, fn="is_inject", inv_freq=None):
    a = dict(a)
    pos = [a.pop(x) for x in ("ids", "preK", "V", "slots", "positions")]
    pk, pv = a.pop("paged_k"), a.pop("paged_v")
    if fn == "is_inject":
        isl.is_inject(*pos, 500000.0, pk, pv, **a)
    elif fn == "is_inject_rotary":
        isl.is_inject_rotary(*pos, 500000.0, pk, pv, inv_freq=inv_freq, **a)
    else:
        ids, preK, V, slots, positions = pos
        m = a.pop("m")
        isl.is_place_inject(ids, preK, V, 500000.0, pk, pv, slots, positions, m,
                            start_pos=3, block_table=T(a["nq"] * 9, i32), page_size=16,
                            max_blocks=9, inv_freq=inv_freq, **a)


@pytest.mark.parametrize("fn", ["is_inject", "is_inject_rotary", "is_place_inject"])
@pytest.mark.parametrize("name,bad,msg", [
    (None, None, "device tensors"),
    ("preK", T(2 * 300 * 2 * 16, torch.int16), "preK must be torch.bfloat16"),
    ("V", T(2 * 300 * 2 * 16 - 1, bf16), "V holds"),
    ("paged_k", T(2 * 128 * 2 * 16 - 8, bf16), "paged_k holds"),
    ("paged_v", T(2 * 128 * 2 * 16, f32), "paged_v must be torch.bfloat16"),
    ("slots", T(80, i32), "slots must be torch.int64"),
    ("positions", T(79, i32), "positions holds 79"),
    ("fact_offsets", T(50, i32), "fact_offsets must be torch.int64"),
    ("fact_lens", T(50, i64), "fact_lens must be torch.int32"),
    ("m", T(2, i64), "m must be torch.int32"),
    ("ids", T(7, i32), "ids holds 7"),
])
def test_inject_family_checks(fn, name, bad, msg):
    a = inject_kw()
    if name:
        a[name] = bad
    with pytest.raises(ValueError, match=msg):
        call_inject(a, fn)


@pytest.mark.parametrize("fn", ["is_inject_rotary", "is_place_inject"])
def test_rotary_table_checks(fn):
    with pytest.raises(ValueError, match="inv_freq must be torch.float64"):
        call_inject(inject_kw(), fn, inv_freq=T(8, f32))
    with pytest.raises(ValueError, match="inv_freq holds 7"):
        call_inject(inject_kw(), fn, inv_freq=T(7, f64))


def test_paged_scores_checks():
    kw = dict(nq=2, Hq=4, H=2, D=16, L=2, num_slots=64, max_blocks=4, max_tokens=30,
              rope_theta=1e4, stream=0)
    good = dict(q=T(2 * 4 * 16, bf16), qpos=T(2, i32), paged_k=T(2 * 64 * 2 * 16, bf16),
                block_table=T(8, i32), m=T(2, i32), scores=T(2 * 4 * 30, f32))

    def call(a):
        isl.is_paged_scores(a["q"], a["qpos"], a["paged_k"], 1, a["block_table"], 16, 0, a["m"],
                            a["scores"], **kw)

    with pytest.raises(ValueError, match="device tensors"):
        call(good)
    for name, bad, msg in [("scores", T(239, f32), "scores holds 239"),
                           ("q", T(128, f32), "q must be torch.bfloat16"),
                           ("qpos", T(2, i64), "qpos must be torch.int32")]:
        a = dict(good, **{name: bad})
        with pytest.raises(ValueError, match=msg):
            call(a)


def test_raw_integers_are_not_pointers():
    a = retrieve_args()
    a["out_ids"] = 1 << 20
    with pytest.raises(TypeError, match="out_ids: expected a torch tensor"):
        call_retrieve(a)
