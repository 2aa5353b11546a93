"""Calls the C ABI must reject on the host, before anything is enqueued.

Each case starts from one valid argument set and breaks one thing.  The
same cases run twice: on host tensors in the CPU suite (status and message;
a rejected call never touches a pointer, so host memory is safe there) and
on device tensors in the GPU suite, where the outputs hold a canary that a
rejected call must leave in place.

The cases call the library through ctypes directly: the Python wrappers
refuse host tensors before the library sees them.
"""
import ctypes

import torch

from paper_2606_01502_amd import mla

CANARY = 7.25  # a value no kernel would write by chance

INVALID = mla.MLA_ERR_INVALID_ARGUMENT
UNSUPPORTED = mla.MLA_ERR_UNSUPPORTED


def _fill(t):
    if t.dtype == torch.float32:
        t.fill_(CANARY)
    return t


def partial_args(device, fp8=False, R=2, Mq=3, H=16, P=8, NB=5, K=3):
    """A valid argument set of mla_sparse_partial_attn_ex (as torch tensors)."""
    kv = torch.uint8 if fp8 else torch.bfloat16
    a = dict(
        q_lat=torch.zeros((R, Mq, H, 512), dtype=torch.bfloat16, device=device),
        q_pe=torch.zeros((R, Mq, H, 64), dtype=torch.bfloat16, device=device),
        ckv=torch.zeros((P, 64, 512), dtype=kv, device=device),
        kpe=torch.zeros((P, 64, 64), dtype=kv, device=device),
        ckv_scale=torch.ones(P, dtype=torch.float32, device=device) if fp8 else None,
        kpe_scale=None,
        table=torch.zeros((R, NB), dtype=torch.int32, device=device),
        sel=torch.zeros((R, K), dtype=torch.int32, device=device),
        scale=0.1,
        out_lat=_fill(torch.empty((R, Mq, H, 512), dtype=torch.float32, device=device)),
        out_lse=_fill(torch.empty((R, Mq, H), dtype=torch.float32, device=device)),
        opts=mla.PartialOpts(),
        tokens=False,
    )
    a["kpe_scale"] = a["ckv_scale"]
    return a


def call_partial(a):
    """Status and last-error text of the partial call with argument set a;
    a descriptor given as the string "null" is passed as a null pointer."""
    lib = mla.load()

    def d(key, scale_key=None):
        t = a[key]
        if isinstance(t, str):
            return None
        return mla.describe(t, a.get(scale_key) if scale_key else None)

    descs = [d("q_lat"), d("q_pe"), d("ckv", "ckv_scale"), d("kpe", "kpe_scale"), d("table"),
             d("sel")]
    outs = [d("out_lat"), d("out_lse")]
    fn = lib.mla_sparse_partial_attn_tokens if a["tokens"] else lib.mla_sparse_partial_attn_ex
    st = fn(*[ctypes.byref(x) if x is not None else None for x in descs],
            ctypes.c_float(a["scale"]),
            *[ctypes.byref(x) if x is not None else None for x in outs],
            ctypes.byref(a["opts"]), ctypes.c_void_p(0))
    return st, lib.mla_last_error().decode()


def _strided_rows(shape, dtype, device, pad):
    """A tensor of `shape` whose rows sit `pad` elements apart beyond their length."""
    base = torch.zeros(shape[:-1] + (shape[-1] + pad,), dtype=dtype, device=device)
    return base[..., :shape[-1]]


def _offset(t, elems):
    """The same shape as t, starting `elems` elements into a larger buffer."""
    flat = torch.zeros(t.numel() + elems, dtype=t.dtype, device=t.device)
    return flat[elems:].view(t.shape)


def _opts(**kw):
    o = mla.PartialOpts()
    for k, v in kw.items():
        if k == "reserved0":
            o.reserved[0] = v
        else:
            setattr(o, k, v)
    return o


# (name, mutation of the argument set, expected status, text the message must contain)
def partial_cases(device):
    f32, bf16, i32 = torch.float32, torch.bfloat16, torch.int32
    z = lambda *s, dt=bf16: torch.zeros(s, dtype=dt, device=device)  # noqa: E731
    cases = []
    for key, word in (("q_lat", "q_lat"), ("q_pe", "q_pe"), ("ckv", "ckv_pool"),
                      ("kpe", "kpe_pool"), ("table", "chunk_block_table"),
                      ("sel", "sel_block_ids"), ("out_lat", "out_lat"), ("out_lse", "out_lse")):
        cases.append((f"null {key}", lambda a, k=key: a.update({k: "null"}), INVALID, word))
    cases += [
        ("q_lat fp32", lambda a: a.update(q_lat=z(2, 3, 16, 512, dt=f32)), INVALID, "q_lat: wrong dtype"),
        ("q_pe fp32", lambda a: a.update(q_pe=z(2, 3, 16, 64, dt=f32)), INVALID, "q_pe: wrong dtype"),
        ("ckv fp32", lambda a: a.update(ckv=z(8, 64, 512, dt=f32)), INVALID, "bf16 or fp8"),
        ("kpe dtype differs", lambda a: a.update(kpe=z(8, 64, 64, dt=torch.uint8)), INVALID,
         "kpe_pool: wrong dtype"),
        ("table fp32", lambda a: a.update(table=z(2, 5, dt=f32)), INVALID, "chunk_block_table: wrong dtype"),
        ("sel int64", lambda a: a.update(sel=z(2, 3, dt=torch.int64)), INVALID, "sel_block_ids: wrong dtype"),
        ("out_lat bf16", lambda a: a.update(out_lat=z(2, 3, 16, 512)), INVALID, "out_lat: wrong dtype"),
        ("out_lse bf16", lambda a: a.update(out_lse=z(2, 3, 16)), INVALID, "out_lse: wrong dtype"),
        ("q_lat 3-d", lambda a: a.update(q_lat=z(6, 16, 512)), INVALID, "q_lat: expected 4 dims"),
        ("out_lse 4-d", lambda a: a.update(out_lse=_fill(z(2, 3, 16, 1, dt=f32))), INVALID,
         "out_lse: expected 3 dims"),
        ("table 3-d", lambda a: a.update(table=z(2, 5, 1, dt=i32)), INVALID, "expected 2 dims"),
        ("sel 1-d", lambda a: a.update(sel=z(3, dt=i32)), INVALID, "sel_block_ids"),
        ("q_lat last dim 511", lambda a: a.update(q_lat=z(2, 3, 16, 511)), INVALID, "512"),
        ("q_pe last dim 63", lambda a: a.update(q_pe=z(2, 3, 16, 63)), INVALID, "q_pe: shape"),
        ("ckv last dim 256", lambda a: a.update(ckv=z(8, 64, 256)), INVALID, "ckv_pool: shape"),
        ("kpe last dim 32", lambda a: a.update(kpe=z(8, 64, 32)), INVALID, "kpe_pool: shape"),
        ("block of 32 tokens", lambda a: a.update(ckv=z(16, 32, 512), kpe=z(16, 32, 64)), INVALID,
         "[P, 64, 512]"),
        ("out_lat last dim 511", lambda a: a.update(out_lat=_fill(z(2, 3, 16, 511, dt=f32))), INVALID,
         "out_lat: shape"),
        ("q_pe R differs", lambda a: a.update(q_pe=z(3, 3, 16, 64)), INVALID, "q_pe: shape"),
        ("out_lat H differs", lambda a: a.update(out_lat=_fill(z(2, 3, 8, 512, dt=f32))), INVALID,
         "out_lat: shape"),
        # jobs come from the table: q's 2 rows must divide them
        ("table R not a multiple of q rows", lambda a: a.update(table=z(3, 5, dt=i32)), INVALID,
         "divide"),
        ("table R twice q rows, sel not", lambda a: a.update(table=z(4, 5, dt=i32)), INVALID,
         "sel_block_ids: shape"),
        ("kpe P differs", lambda a: a.update(kpe=z(9, 64, 64)), INVALID, "kpe_pool: shape"),
        ("q_lat inner stride 2", lambda a: a.update(q_lat=z(2, 3, 16, 1024)[..., ::2]), INVALID,
         "innermost stride"),
        ("q_lat base misaligned", lambda a: a.update(q_lat=_offset(a["q_lat"], 1)), INVALID,
         "16-byte aligned"),
        ("q_pe rows misaligned", lambda a: a.update(q_pe=_strided_rows((2, 3, 16, 64), bf16, device, 2)),
         INVALID, "16-byte aligned"),
        ("out_lat rows misaligned",
         lambda a: a.update(out_lat=_fill(_strided_rows((2, 3, 16, 512), f32, device, 1))), INVALID,
         "out_lat rows must be 16-byte aligned"),
        ("ckv pool strided", lambda a: a.update(ckv=z(16, 64, 512)[::2]), INVALID, "contiguous"),
        ("out_lat aliases q_lat", lambda a: a.update(out_lat=_alias_out_on_q(a)), INVALID, "overlap"),
        ("out_lse inside out_lat", lambda a: a.update(out_lse=a["out_lat"].view(-1)[1000:1096].view(2, 3, 16)),
         INVALID, "overlap"),
        ("out_lse overlaps sel", lambda a: a.update(out_lse=_lse_on_sel(a)), INVALID, "overlap"),
        ("scale inf", lambda a: a.update(scale=float("inf")), INVALID, "scale"),
        ("scale nan", lambda a: a.update(scale=float("nan")), INVALID, "scale"),
        ("scale just above 2^64", lambda a: a.update(scale=2.0 ** 64 * (1 + 2.0 ** -23)), INVALID,
         "2^64"),
        ("scale -2^65", lambda a: a.update(scale=-(2.0 ** 65)), INVALID, "2^64"),
        ("opts reserved", lambda a: a.update(opts=_opts(reserved0=1)), INVALID, "reserved"),
        ("opts n_splits -1", lambda a: a.update(opts=_opts(n_splits=-1)), INVALID, "n_splits"),
        ("opts row_tile 96", lambda a: a.update(opts=_opts(row_tile=96)), INVALID, "row_tile"),
        ("block_scale on a bf16 pool", lambda a: a.update(ckv_scale=torch.ones(8, dtype=f32, device=device)),
         INVALID, "block_scale must be NULL"),
        ("per-row sel Mq differs", lambda a: a.update(sel=z(2, 4, 3, dt=i32)), INVALID, "[R, Mq, K]"),
        ("token sel 3-d", lambda a: a.update(sel=z(2, 3, 3, dt=i32), tokens=True), INVALID,
         "sel_token_ids"),
        ("per-row NB x rows too large", lambda a: a.update(sel=z(2, 3, 3, dt=i32), table=z(2, 40000, dt=i32)),
         UNSUPPORTED, "NB"),
    ]
    return cases


def partial_cases_fp8(device):
    return [
        ("fp8 without any block_scale", lambda a: a.update(ckv_scale=None, kpe_scale=None), INVALID,
         "block_scale"),
        ("fp8 kpe without block_scale", lambda a: a.update(kpe_scale=None), INVALID, "block_scale"),
        ("fp8 scale inf", lambda a: a.update(scale=float("inf")), INVALID, "scale"),
        ("fp8 kpe bf16", lambda a: a.update(kpe=torch.zeros((8, 64, 64), dtype=torch.bfloat16,
                                                            device=device)), INVALID, "kpe_pool"),
        ("fp8 out_lse on the scales", lambda a: a.update(out_lse=_lse_on_scales(a)), INVALID, "overlap"),
    ]


def _alias_out_on_q(a):
    """Moves q_lat into the first part of a byte buffer and returns an fp32
    out_lat view that starts in the middle of q_lat's bytes."""
    q, out = a["q_lat"], a["out_lat"]
    n_q, n_out = q.numel() * 2, out.numel() * 4
    buf = torch.zeros(n_q // 2 + n_out, dtype=torch.uint8, device=q.device)
    a["q_lat"] = buf[:n_q].view(torch.bfloat16).view(q.shape)
    return _fill(buf[n_q // 2:n_q // 2 + n_out].view(torch.float32).view(out.shape))


def _lse_on_sel(a):
    """Moves sel into an int32 buffer and returns an out_lse view whose first
    element is sel's last."""
    sel, lse = a["sel"], a["out_lse"]
    buf = torch.zeros(sel.numel() - 1 + lse.numel(), dtype=torch.int32, device=sel.device)
    a["sel"] = buf[:sel.numel()].view(sel.shape)
    return _fill(buf[sel.numel() - 1:].view(torch.float32).view(lse.shape))


def _lse_on_scales(a):
    """Moves the fp8 block scales into a float buffer and returns an out_lse
    view over its last two scales and beyond."""
    sc, lse = a["ckv_scale"], a["out_lse"]
    buf = torch.ones(sc.numel() - 2 + lse.numel(), dtype=torch.float32, device=sc.device)
    a["ckv_scale"] = a["kpe_scale"] = buf[:sc.numel()]
    return _fill(buf[sc.numel() - 2:].view(lse.shape))


# ------------------------------------------------------------------ merge
def merge_args(device, n=3, B=2, Mq=1, H=8):
    return dict(
        lat=[torch.zeros((B, Mq, H, 512), dtype=torch.float32, device=device) for _ in range(n)],
        lse=[torch.zeros((B, Mq, H), dtype=torch.float32, device=device) for _ in range(n)],
        out=_fill(torch.empty((B, Mq, H, 512), dtype=torch.float32, device=device)),
        out_lse=_fill(torch.empty((B, Mq, H), dtype=torch.float32, device=device)),
        n=n, null_arrays=False)


def call_merge(a):
    lib = mla.load()
    d_lat = [mla.describe(t) for t in a["lat"]]
    d_lse = [mla.describe(t) for t in a["lse"]]
    k = max(len(d_lat), 1)
    arr_lat = (ctypes.POINTER(mla.Tensor) * k)(*[ctypes.pointer(x) for x in d_lat])
    arr_lse = (ctypes.POINTER(mla.Tensor) * k)(*[ctypes.pointer(x) for x in d_lse])
    d_out = mla.describe(a["out"]) if not isinstance(a["out"], str) else None
    d_ol = mla.describe(a["out_lse"]) if a["out_lse"] is not None else None
    st = lib.mla_merge_partials_ex(None if a["null_arrays"] else arr_lat,
                                   None if a["null_arrays"] else arr_lse, int(a["n"]),
                                   ctypes.byref(d_out) if d_out is not None else None,
                                   ctypes.byref(d_ol) if d_ol is not None else None,
                                   ctypes.c_void_p(0))
    return st, lib.mla_last_error().decode()


def merge_cases(device):
    f32 = torch.float32
    z = lambda *s: torch.zeros(s, dtype=f32, device=device)  # noqa: E731
    many = lambda a, n: a.update(lat=[a["lat"][0]] * n, lse=[a["lse"][0]] * n, n=n)  # noqa: E731
    return [
        ("n_parts 0", lambda a: a.update(n=0), INVALID, "n_parts"),
        ("n_parts 65", lambda a: many(a, 65), INVALID, "n_parts"),
        ("n_parts -1", lambda a: a.update(n=-1), INVALID, "n_parts"),
        ("null part arrays", lambda a: a.update(null_arrays=True), INVALID, "null part arrays"),
        ("null out", lambda a: a.update(out="null"), INVALID, "out: null descriptor"),
        ("part shape differs", lambda a: a["lat"].__setitem__(1, z(2, 1, 4, 512)), INVALID,
         "shape of out"),
        ("part lse shape differs", lambda a: a["lse"].__setitem__(2, z(2, 1, 9)), INVALID,
         "out_lse parts"),
        ("part strides differ", lambda a: a["lat"].__setitem__(1, _strided_rows((2, 1, 8, 512), f32,
                                                                                device, 4)),
         UNSUPPORTED, "strides"),
        # part 0's dtype picks the form (fp32, or the bf16 wire form): a bf16
        # part after an fp32 one mixes the two
        ("parts mix fp32 and bf16", lambda a: a["lat"].__setitem__(1, torch.zeros((2, 1, 8, 512),
                                                                                  dtype=torch.bfloat16,
                                                                                  device=device)),
         INVALID, "wrong dtype"),
        ("wire part with a [B, Mq, H] lse", lambda a: a["lat"].__setitem__(
            0, torch.zeros((2, 1, 8, 512), dtype=torch.bfloat16, device=device)), INVALID,
         "expected 4 dims"),
        ("out last dim 511", lambda a: a.update(out=_fill(z(2, 1, 8, 511))), INVALID, "512"),
        ("out rows misaligned", lambda a: a.update(out=_fill(_strided_rows((2, 1, 8, 512), f32, device, 2))),
         INVALID, "16-byte aligned"),
        ("out is a part", lambda a: a.update(out=a["lat"][1]), INVALID, "overlaps"),
        ("merged lse on a part's lse", lambda a: a.update(out_lse=a["lse"][0]), INVALID, "overlaps"),
        ("merged lse shape", lambda a: a.update(out_lse=_fill(z(2, 1, 4))), INVALID, "merged_lse"),
    ]
