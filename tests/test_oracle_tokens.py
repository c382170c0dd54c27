"""Pins of the oracle's per-token encryption (GIFT Sec. 4.5) -- no GPU.

Each non-EOS token's ciphertext must equal OpenSSL's AES-256 of
LE64(token) || LE64(nonce) under the owner's key; the EOS token maps to the
reserved all-0xFF block for every key; decryption recovers token and nonce.
"""
import numpy as np
import pytest

import oracle
import openssl_ref

pytestmark = pytest.mark.skipif(not openssl_ref.available(), reason="libcrypto not available")

rng = np.random.default_rng(99)
EOS = 128001


def setup(n_users=4, n_tokens=40):
    keys = rng.integers(0, 256, (n_users, 32), dtype=np.uint8)
    tok = rng.integers(0, 128256, n_tokens).astype(np.uint64)
    non = rng.integers(0, 2**63, n_tokens).astype(np.uint64) * np.uint64(2) + np.uint64(1)
    return keys, tok, non


def test_blocks_match_openssl_and_eos_is_reserved():
    keys, tok, non = setup()
    tok[[3, 17]] = EOS
    segs = [(0, 10, 0, 0), (12, 20, 3, 0), (32, 8, 1, 0)]
    st, out = oracle.token_encrypt(segs, tok, non, keys, EOS)
    assert st == 0
    for b, c, u, _ in segs:
        for r in range(b, b + c):
            if tok[r] == EOS:
                assert out[r].tobytes() == b"\xff" * 16
            else:
                blk = int(tok[r]).to_bytes(8, "little") + int(non[r]).to_bytes(8, "little")
                assert out[r].tobytes() == openssl_ref.aes256_ecb_encrypt(keys[u].tobytes(), blk)
    for r in (10, 11):  # uncovered
        assert not out[r].any()


def test_round_trip_recovers_tokens_and_nonces():
    keys, tok, non = setup()
    tok[5] = EOS
    segs = [(0, 40, 2, 0)]
    _, out = oracle.token_encrypt(segs, tok, non, keys, EOS)
    st, t2, n2 = oracle.token_decrypt(segs, out, keys, EOS)
    assert st == 0 and (t2 == tok).all()
    mask = tok != EOS
    assert (n2[mask] == non[mask]).all() and n2[5] == 0


def test_nonces_hide_repeated_tokens():
    keys, tok, non = setup()
    tok[:] = 42
    _, out = oracle.token_encrypt([(0, 40, 0, 0)], tok, non, keys, EOS)
    assert len({o.tobytes() for o in out}) == 40
    # same token and nonce under another user's key differs too
    _, out2 = oracle.token_encrypt([(0, 40, 1, 0)], tok, non, keys, EOS)
    assert all(a.tobytes() != b.tobytes() for a, b in zip(out, out2))


def test_wrong_owner_gives_unrelated_tokens():
    keys, tok, non = setup()
    _, out = oracle.token_encrypt([(0, 40, 0, 0)], tok, non, keys, EOS)
    _, t2, _ = oracle.token_decrypt([(0, 40, 1, 0)], out, keys, EOS)
    assert (t2 != tok).all()
    assert (t2 >= 128256).mean() > 0.99  # almost surely outside the vocabulary


def test_validation():
    keys, tok, non = setup()
    assert oracle.token_encrypt([(0, 0, 0, 0)], tok, non, keys, EOS)[0] == oracle.E_INVALID
    assert oracle.token_encrypt([(39, 2, 0, 0)], tok, non, keys, EOS)[0] == oracle.E_RANGE
    assert oracle.token_encrypt([(0, 2, 4, 0)], tok, non, keys, EOS)[0] == oracle.E_RANGE
    assert oracle.token_encrypt([(0, 2, 0, 0), (1, 2, 1, 0)], tok, non, keys, EOS)[0] == oracle.E_OVERLAP
    # iv_seq is not used: equal (user, iv_seq) pairs are fine
    assert oracle.token_encrypt([(0, 2, 0, 7), (2, 2, 0, 7)], tok, non, keys, EOS)[0] == 0
