"""Pins of the CPU oracle to facts outside itself (no GPU).

AES-256 (FIPS-197) and GCM (SP 800-38D) are pinned by:
  - algebraic properties of the S-box and of GF(2^128) that follow from the
    definitions (bijectivity, no fixed points, field axioms, x * x^127 =
    x^128 = 1 + x + x^2 + x^7, the Frobenius map H^(2^128) = H);
  - OpenSSL's independent AES-256 and AES-256-GCM on random inputs and on
    lengths from 0 to over 1 MiB, including every partial-block length;
  - exhaustive single-bit tampering of short messages.
The published FIPS-197/GCM known-answer vectors are not in this offline
environment and are not typed in from memory; OpenSSL stands in for them.
"""
import os

import numpy as np
import pytest

import oracle
import openssl_ref

pytestmark = pytest.mark.skipif(not openssl_ref.available(), reason="libcrypto not available")

rng = np.random.default_rng(20260)


def rbytes(n):
    return rng.integers(0, 256, n, dtype=np.uint8).tobytes()


# --------------------------------------------------------------------------
# AES
# --------------------------------------------------------------------------
def test_sbox_is_a_bijection_without_fixed_or_opposite_fixed_points():
    s, inv = oracle.sbox()
    assert sorted(s.tolist()) == list(range(256))
    assert all(int(inv[s[x]]) == x for x in range(256))
    # the affine constant was chosen so that S(x) != x and S(x) != ~x
    assert all(int(s[x]) != x for x in range(256))
    assert all(int(s[x]) != (x ^ 0xFF) for x in range(256))
    # S(0) = affine(0) = the affine constant
    assert int(s[0]) == 0x63


def test_sbox_is_affine_image_of_field_inverse():
    # S(a) xor S(0) is GF(2)-linear in inverse(a): check linearity on pairs via
    # a brute-force inverse in GF(2^8) computed here from the field polynomial
    def mul(a, b):
        p = 0
        for _ in range(8):
            if b & 1:
                p ^= a
            hi = a & 0x80
            a = (a << 1) & 0xFF
            if hi:
                a ^= 0x1B
            b >>= 1
        return p

    inv = [0] * 256
    for a in range(1, 256):
        inv[a] = next(b for b in range(1, 256) if mul(a, b) == 1)
    s, _ = oracle.sbox()
    lin = {inv[a]: int(s[a]) ^ 0x63 for a in range(256)}
    for u in range(0, 256, 7):
        for v in range(0, 256, 11):
            assert lin[u ^ v] == lin[u] ^ lin[v]


def test_aes256_matches_openssl_on_random_blocks():
    for _ in range(400):
        k, b = rbytes(32), rbytes(16)
        assert oracle.aes_encrypt_block(k, b) == openssl_ref.aes256_ecb_encrypt(k, b)


def test_aes256_special_keys_match_openssl():
    for k in (bytes(32), b"\xff" * 32, bytes(range(32))):
        for b in (bytes(16), b"\xff" * 16, bytes(range(16))):
            assert oracle.aes_encrypt_block(k, b) == openssl_ref.aes256_ecb_encrypt(k, b)


def test_inverse_cipher_inverts():
    for _ in range(200):
        k, b = rbytes(32), rbytes(16)
        assert oracle.aes_decrypt_block(k, oracle.aes_encrypt_block(k, b)) == b


def test_key_expansion_first_words_are_the_key():
    k = rbytes(32)
    w = oracle.key_expansion(k)
    assert w[:32].tobytes() == k


# --------------------------------------------------------------------------
# GF(2^128)
# --------------------------------------------------------------------------
def elem(p):
    """x^p in GCM bit order (bit 0 = MSB of byte 0)."""
    b = bytearray(16)
    b[p // 8] = 0x80 >> (p % 8)
    return bytes(b)


ONE = elem(0)


def xor(a, b):
    return bytes(x ^ y for x, y in zip(a, b))


def test_gf_identity_and_zero():
    for _ in range(50):
        a = rbytes(16)
        assert oracle.gf128_mul(a, ONE) == a
        assert oracle.gf128_mul(ONE, a) == a
        assert oracle.gf128_mul(a, bytes(16)) == bytes(16)


def test_gf_reduction_closed_form():
    # x * x^127 = x^128 = 1 + x + x^2 + x^7 (the GCM field polynomial)
    expect = xor(xor(elem(0), elem(1)), xor(elem(2), elem(7)))
    assert oracle.gf128_mul(elem(1), elem(127)) == expect
    # products below degree 128 are plain shifts
    for i in range(0, 128, 9):
        for j in range(0, 128 - i, 13):
            assert oracle.gf128_mul(elem(i), elem(j)) == elem(i + j)


def test_gf_field_axioms():
    for _ in range(60):
        a, b, c = rbytes(16), rbytes(16), rbytes(16)
        assert oracle.gf128_mul(a, b) == oracle.gf128_mul(b, a)
        assert oracle.gf128_mul(oracle.gf128_mul(a, b), c) == oracle.gf128_mul(a, oracle.gf128_mul(b, c))
        assert oracle.gf128_mul(a, xor(b, c)) == xor(oracle.gf128_mul(a, b), oracle.gf128_mul(a, c))


def test_gf_frobenius():
    # in GF(2^128), h^(2^128) = h: 128 squarings return to the start only if the
    # multiply implements a field of exactly 2^128 elements
    for _ in range(3):
        h = rbytes(16)
        y = h
        for _ in range(128):
            y = oracle.gf128_mul(y, y)
        assert y == h


def test_ghash_is_linear_and_horner():
    h = rbytes(16)
    a, b = rbytes(64), rbytes(64)
    assert oracle.ghash(h, xor(a, b)) == xor(oracle.ghash(h, a), oracle.ghash(h, b))
    # one block: X1 * H
    x = rbytes(16)
    assert oracle.ghash(h, x) == oracle.gf128_mul(x, h)
    # two blocks: X1*H^2 + X2*H
    x2 = rbytes(16)
    h2 = oracle.gf128_mul(h, h)
    assert oracle.ghash(h, x + x2) == xor(oracle.gf128_mul(x, h2), oracle.gf128_mul(x2, h))


# --------------------------------------------------------------------------
# GCM
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n", list(range(0, 65)) + [255, 256, 257, 4095, 4096 + 3, 65536 + 3])
def test_gcm_matches_openssl(n):
    k, iv, p = rbytes(32), rbytes(12), rbytes(n)
    assert oracle.gcm_encrypt(k, iv, p) == openssl_ref.gcm_encrypt(k, iv, p)


def test_gcm_long_message_matches_openssl():
    k, iv, p = rbytes(32), rbytes(12), rbytes((1 << 20) + 5)
    assert oracle.gcm_encrypt(k, iv, p) == openssl_ref.gcm_encrypt(k, iv, p)


def test_gcm_roundtrip_and_openssl_accepts_oracle_tag():
    for n in (0, 1, 15, 16, 17, 100, 1000):
        k, iv, p = rbytes(32), rbytes(12), rbytes(n)
        c, t = oracle.gcm_encrypt(k, iv, p)
        assert oracle.gcm_decrypt(k, iv, c, t) == p
        assert openssl_ref.gcm_decrypt(k, iv, c, t) == p


@pytest.mark.parametrize("n", [1, 16, 17, 33, 48])
def test_gcm_every_single_bit_flip_fails(n):
    k, iv, p = rbytes(32), rbytes(12), rbytes(n)
    c, t = oracle.gcm_encrypt(k, iv, p)
    for i in range(8 * n):
        cc = bytearray(c)
        cc[i // 8] ^= 1 << (i % 8)
        assert oracle.gcm_decrypt(k, iv, bytes(cc), t) is None
    for i in range(128):
        tt = bytearray(t)
        tt[i // 8] ^= 1 << (i % 8)
        assert oracle.gcm_decrypt(k, iv, c, bytes(tt)) is None


def test_gcm_counter_increment_wraps_in_low_32_bits():
    # an IV whose derived counters cross the 2^32 boundary would use inc32's
    # wrap; with 96-bit IVs J0 ends in ...0001, so counters 2.. never wrap for
    # legal lengths -- check that consecutive blocks use consecutive counters
    k, iv = rbytes(32), rbytes(12)
    p = bytes(48)
    c, _ = oracle.gcm_encrypt(k, iv, p)
    for j in range(3):
        cb = iv + (2 + j).to_bytes(4, "big")
        assert c[16 * j:16 * j + 16] == openssl_ref.aes256_ecb_encrypt(k, cb)
