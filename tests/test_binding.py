"""The Python binding checks every tensor against the layout include/locks.h
documents before anything reaches the library (CPU tensors: the checks run before
the device check, and nothing is launched)."""
import pytest
import torch

from paper_2607_24555_amd import locks as B


def _cfg(**kw):
    c = B.Config(num_seqs=2, num_q_heads=8, num_kv_heads=2, rank=8, budget_tokens=256,
                 max_pages_per_seq=10, num_blocks=20)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def _args(cfg):
    S, Hq, Hkv, mp, nb = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.max_pages_per_seq, cfg.num_blocks
    dt = torch.bfloat16 if cfg.kv_dtype == B.LOCKS_BF16 else torch.float32
    return dict(
        q=torch.zeros(S, Hq, 128, dtype=torch.bfloat16 if cfg.q_dtype == B.LOCKS_BF16 else torch.float32),
        k=torch.zeros(nb, Hkv, cfg.page_size, 128, dtype=dt),
        v=torch.zeros(nb, Hkv, cfg.page_size, 128, dtype=dt),
        pt=torch.zeros(S, mp, dtype=torch.int32), sl=torch.zeros(S, dtype=torch.int32),
        summ=torch.zeros(nb, Hkv, B.summary_stride(cfg.rank, cfg.basis), dtype=torch.uint8),
        ws=torch.zeros(1024, dtype=torch.uint8))


def _step(cfg, a, **over):
    a = dict(a, **over)
    return B.decode_step(cfg, a["q"], a["k"], a["v"], a["pt"], a["sl"], a["summ"], a["ws"],
                         build_list=a.get("bl"), out_ids=a.get("ids"), out_sel_lse=a.get("sel"),
                         out=a.get("out"), out_lse=a.get("lse"), k_new=a.get("kn"),
                         v_new=a.get("vn"))


@pytest.mark.parametrize("what,bad,msg", [
    ("q", lambda c: torch.zeros(2, 8, 128, dtype=torch.float32), "q: dtype"),
    ("q", lambda c: torch.zeros(2, 4, 128, dtype=torch.bfloat16), "q: shape"),
    ("k", lambda c: torch.zeros(20, 2, 16, 128, dtype=torch.float32), "k_cache: dtype"),
    ("v", lambda c: torch.zeros(19, 2, 16, 128, dtype=torch.bfloat16), "v_cache: shape"),
    ("pt", lambda c: torch.zeros(2, 10, dtype=torch.int64), "page_table: dtype"),
    ("sl", lambda c: torch.zeros(3, dtype=torch.int32), "seq_lens: shape"),
    ("summ", lambda c: torch.zeros(20, 2, 818, dtype=torch.uint8), "summaries: shape"),
    ("bl", lambda c: torch.zeros(4, 2, dtype=torch.int64), "build_list"),
    ("bl", lambda c: torch.zeros(4, 3, dtype=torch.int32), "build_list"),
    ("ids", lambda c: torch.zeros(2, 2, 15, dtype=torch.int32), "out_ids: shape"),
    ("sel", lambda c: torch.zeros(2, 8, 16, dtype=torch.float16), "out_sel_lse: dtype"),
    ("out", lambda c: torch.zeros(2, 8, 64, dtype=torch.float32), "out: shape"),
    ("lse", lambda c: torch.zeros(2, 2, dtype=torch.float32), "out_lse: shape"),
    ("kn", lambda c: torch.zeros(2, 2, 128, dtype=torch.float32), "k_new: dtype"),
    ("ws", lambda c: torch.zeros(256, dtype=torch.int32), "ws"),
])
def test_decode_step_rejects_mismatched_tensors(what, bad, msg):
    cfg = _cfg()
    a = _args(cfg)
    a["ids"], a["sel"] = torch.zeros(2, 2, 16, dtype=torch.int32), torch.zeros(2, 8, 16)
    a["out"], a["lse"] = torch.zeros(2, 8, 128), torch.zeros(2, 8)
    a[what] = bad(cfg)
    with pytest.raises(B.LocksError, match=msg):
        _step(cfg, a)


def test_well_formed_host_tensors_reach_the_device_check():
    cfg = _cfg()
    a = _args(cfg)
    a["ids"], a["sel"] = torch.zeros(2, 2, 16, dtype=torch.int32), torch.zeros(2, 8, 16)
    a["out"], a["lse"] = torch.zeros(2, 8, 128), torch.zeros(2, 8)
    with pytest.raises(B.LocksError, match="device tensors"):
        _step(cfg, a)


def test_other_calls_check_their_tensors():
    cfg = _cfg(kv_dtype=B.LOCKS_FP32, q_dtype=B.LOCKS_FP32)
    a = _args(cfg)
    with pytest.raises(B.LocksError, match="k_cache: dtype"):
        B.build_summaries(cfg, a["k"].bfloat16(), a["pt"], a["sl"], a["summ"])
    with pytest.raises(B.LocksError, match="page_ids: shape"):
        B.sparse_attend(cfg, a["q"], a["k"], a["v"], a["pt"], a["sl"],
                        torch.zeros(2, 2, 3, dtype=torch.int32), a["ws"],
                        out=torch.zeros(2, 8, 128), out_lse=torch.zeros(2, 8))
    with pytest.raises(B.LocksError, match="out_all_lse: shape"):
        B.score_pages(cfg, a["q"], a["summ"], a["pt"], a["sl"], a["ws"], torch.zeros(2, 8, 9))
    with pytest.raises(B.LocksError, match="seq_lens: dtype"):
        B.dense_attend(cfg, a["q"], a["k"], a["v"], a["pt"], a["sl"].long(), a["ws"],
                       out=torch.zeros(2, 8, 128), out_lse=torch.zeros(2, 8))
    with pytest.raises(B.LocksError, match="v_new: shape"):
        B.append_kv(cfg, torch.zeros(2, 2, 128), torch.zeros(2, 1, 128), a["k"], a["v"], a["pt"],
                    a["sl"])
    with pytest.raises(B.LocksError, match="page_list"):
        B.kivi_quantize(cfg, B.Kivi(4, 32, 0), a["k"], a["v"], a["pt"], a["sl"],
                        torch.zeros(3, dtype=torch.int32))
