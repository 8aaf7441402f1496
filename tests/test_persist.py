"""Persistence and reading back of checkpoints (Sec. 4.4.3, Sec. 4.3.2):
host-only library calls, no GPU."""
import os

import numpy as np
import pytest

from paper_2511_07035_amd import (GockptError, gockpt_find_latest_checkpoint, gockpt_read_checkpoint,
                                  gockpt_read_checkpoint_info, gockpt_read_checkpoint_user, gockpt_write_checkpoint)


def _arrays(n, seed):
    rng = np.random.default_rng(seed)
    bits = rng.integers(0, 1 << 32, size=(3, n), dtype=np.uint64).astype(np.uint32)
    special = np.array([0x00000000, 0x80000000, 0x00000001, 0x807FFFFF, 0x7F800000, 0xFF800000, 0x7FC00001,
                        0xFFFFFFFF], dtype=np.uint32)
    k = min(n, special.size)
    bits[:, :k] = special[:k]
    return [b.view(np.float32) for b in bits]


def _crc_line(path, name):
    for line in open(os.path.join(path, "meta")):
        if line.startswith(name + " "):
            return line.split()[1].split(",")
    raise KeyError(name)


@pytest.mark.parametrize("n,piece,threads", [(0, 4096, 1), (1, 4096, 2), (1023, 4096, 3), (100_003, 4096, 8),
                                             (100_003, 0, 0)])
def test_roundtrip_bitwise(tmp_path, n, piece, threads):
    p, m, v = _arrays(n, n)
    d = str(tmp_path / "ck")
    st = gockpt_write_checkpoint(d, p, m, v, t=123, tracker=7, scale=32768.0, K=8, skipped=2, beta1=0.9,
                                 beta2=0.95, eps=1e-8, weight_decay=0.1, nthreads=threads, piece_bytes=piece)
    assert st.bytes == 12 * n
    q, r, s, info, _ = gockpt_read_checkpoint(d, n, nthreads=threads)
    for a, b in ((p, q), (m, r), (v, s)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert (info.n, info.t, info.tracker, info.scale, info.K, info.skipped) == (n, 123, 7, 32768.0, 8, 2)
    assert (info.beta1, info.beta2, info.eps, info.weight_decay) == (0.9, 0.95, 1e-8, 0.1)  # exact (hex floats)
    assert os.path.getsize(os.path.join(d, "data.bin")) == info.data_bytes


def test_crc32c_matches_the_iscsi_test_vectors(tmp_path):
    """The per-piece checksum is CRC-32C; the three 32-byte vectors of RFC 3720
    (B.4): all zeros, all ones, bytes 0..31 ascending."""
    zeros = np.zeros(8, np.uint32).view(np.float32)
    ones = np.full(8, 0xFFFFFFFF, np.uint32).view(np.float32)
    asc = np.arange(32, dtype=np.uint8).view(np.uint32).view(np.float32)
    d = str(tmp_path / "v")
    gockpt_write_checkpoint(d, zeros, ones, asc.copy())
    assert _crc_line(d, "crc_master") == ["8a9136aa"]
    assert _crc_line(d, "crc_exp_avg") == ["62a8ab43"]
    assert _crc_line(d, "crc_exp_avg_sq") == ["46dd794e"]


def test_metadata_is_the_commit_point(tmp_path):
    """Without `meta` a checkpoint does not exist: reading fails and the
    latest-checkpoint search passes over it."""
    root = tmp_path / "run"
    root.mkdir()
    n = 4096
    for t in (5, 9, 7):
        p, m, v = _arrays(n, t)
        gockpt_write_checkpoint(str(root / f"step{t}"), p, m, v, t=t)
    p, m, v = _arrays(n, 12)
    gockpt_write_checkpoint(str(root / "step12"), p, m, v, t=12)
    assert gockpt_find_latest_checkpoint(str(root)).endswith("step12")
    os.unlink(root / "step12" / "meta")  # a crash before the metadata was committed
    with pytest.raises(GockptError, match="meta missing"):
        gockpt_read_checkpoint(str(root / "step12"), n)
    assert gockpt_find_latest_checkpoint(str(root)).endswith("step9")
    (root / "not_a_ckpt").mkdir()
    assert gockpt_find_latest_checkpoint(str(root)).endswith("step9")
    with pytest.raises(GockptError):
        gockpt_find_latest_checkpoint(str(tmp_path / "empty_missing"))


def test_rewriting_a_directory_replaces_it(tmp_path):
    d = str(tmp_path / "ck")
    a = _arrays(5000, 1)
    b = _arrays(5000, 2)
    gockpt_write_checkpoint(d, *a, t=1)
    gockpt_write_checkpoint(d, *b, t=2, piece_bytes=8192)
    q, r, s, info, _ = gockpt_read_checkpoint(d, 5000)
    assert info.t == 2 and np.array_equal(q.view(np.uint32), b[0].view(np.uint32))
    assert not os.path.exists(os.path.join(d, "meta.tmp"))
    assert sorted(os.listdir(tmp_path)) == ["ck"]  # no sibling left behind


def test_a_failed_rewrite_keeps_the_previous_checkpoint(tmp_path):
    """The new checkpoint is written beside the old one and put in place only
    when complete (Sec. 4.4.3 persistence): when writing it fails -- here its
    sibling work directory cannot be made -- the directory still holds the
    previous complete checkpoint, and a rewrite after the obstacle is gone
    succeeds."""
    d = str(tmp_path / "ck")
    a = _arrays(3000, 1)
    gockpt_write_checkpoint(d, *a, t=1, user_meta="first\n")
    blocker = tmp_path / "ck.gockpt-tmp" / "occupied"
    blocker.mkdir(parents=True)  # a non-empty directory where the work directory would go
    with pytest.raises(GockptError, match="mkdir"):
        gockpt_write_checkpoint(d, *_arrays(3000, 2), t=2)
    q, r, s, info, _ = gockpt_read_checkpoint(d, 3000)
    assert info.t == 1 and np.array_equal(q.view(np.uint32), a[0].view(np.uint32))
    assert gockpt_read_checkpoint_user(d) == "first\n"
    blocker.rmdir()
    gockpt_write_checkpoint(d, *_arrays(3000, 3), t=3)
    assert gockpt_read_checkpoint_info(d).t == 3
    assert gockpt_find_latest_checkpoint(str(tmp_path)).endswith("ck")


@pytest.mark.parametrize("where", [0, 1, 2])
def test_corruption_is_detected(tmp_path, where):
    n = 50_000
    d = str(tmp_path / "ck")
    gockpt_write_checkpoint(d, *_arrays(n, 3), piece_bytes=16384)
    info = gockpt_read_checkpoint_info(d)
    stride = (4 * n + 4095) // 4096 * 4096
    with open(os.path.join(d, "data.bin"), "r+b") as f:
        f.seek(where * stride + 4 * 31_337)
        byte = f.read(1)
        f.seek(where * stride + 4 * 31_337)
        f.write(bytes([byte[0] ^ 0x10]))
    name = ["master", "exp_avg", "exp_avg_sq"][where]
    with pytest.raises(GockptError, match=f"checksum mismatch in {name} at byte"):
        gockpt_read_checkpoint(d, n)
    assert info.n == n


def test_truncated_and_mismatched(tmp_path):
    n = 20_000
    d = str(tmp_path / "ck")
    gockpt_write_checkpoint(d, *_arrays(n, 4))
    with pytest.raises(GockptError, match="elements"):
        gockpt_read_checkpoint(d, n + 8)
    os.truncate(os.path.join(d, "data.bin"), 4 * n)
    with pytest.raises(GockptError, match="shorter"):
        gockpt_read_checkpoint(d, n)


def test_user_text_roundtrip(tmp_path):
    d = str(tmp_path / "ck")
    text = "step 4000\ntokens/s 794.1\nwall 3600.5 s\nnote: ünïcödé\n"
    gockpt_write_checkpoint(d, *_arrays(64, 5), user_meta=text)
    assert gockpt_read_checkpoint_info(d).has_user == 1
    assert gockpt_read_checkpoint_user(d) == text
    d2 = str(tmp_path / "ck2")
    gockpt_write_checkpoint(d2, *_arrays(64, 6))
    assert gockpt_read_checkpoint_user(d2) == ""


def test_bad_arguments(tmp_path):
    p, m, v = _arrays(100, 7)
    with pytest.raises(GockptError):
        gockpt_write_checkpoint(str(tmp_path / "x"), p, m, v, piece_bytes=1000)  # not a multiple of 4096
    with pytest.raises(GockptError):
        gockpt_read_checkpoint_info(str(tmp_path / "nowhere"))
    with pytest.raises(ValueError):
        gockpt_write_checkpoint(str(tmp_path / "y"), p, m[:50], v)
