"""OpenSSL's AES-256 and AES-256-GCM through ctypes: an independent
implementation used to pin the CPU oracle.  Tests only."""
import ctypes
import ctypes.util

_crypto = None
EVP_CTRL_AEAD_SET_IVLEN = 0x9
EVP_CTRL_AEAD_GET_TAG = 0x10
EVP_CTRL_AEAD_SET_TAG = 0x11


def available():
    try:
        _lib()
        return True
    except OSError:
        return False


def _lib():
    global _crypto
    if _crypto is None:
        name = ctypes.util.find_library("crypto") or "libcrypto.so.3"
        L = ctypes.CDLL(name)
        P = ctypes.c_void_p
        L.EVP_CIPHER_CTX_new.restype = P
        L.EVP_CIPHER_CTX_free.argtypes = [P]
        L.EVP_aes_256_gcm.restype = P
        L.EVP_aes_256_ecb.restype = P
        L.EVP_EncryptInit_ex.argtypes = [P, P, P, P, P]
        L.EVP_DecryptInit_ex.argtypes = [P, P, P, P, P]
        L.EVP_EncryptUpdate.argtypes = [P, P, ctypes.POINTER(ctypes.c_int), P, ctypes.c_int]
        L.EVP_DecryptUpdate.argtypes = [P, P, ctypes.POINTER(ctypes.c_int), P, ctypes.c_int]
        L.EVP_EncryptFinal_ex.argtypes = [P, P, ctypes.POINTER(ctypes.c_int)]
        L.EVP_DecryptFinal_ex.argtypes = [P, P, ctypes.POINTER(ctypes.c_int)]
        L.EVP_CIPHER_CTX_ctrl.argtypes = [P, ctypes.c_int, ctypes.c_int, P]
        L.EVP_CIPHER_CTX_set_padding.argtypes = [P, ctypes.c_int]
        _crypto = L
    return _crypto


def aes256_ecb_encrypt(key, block):
    L = _lib()
    ctx = L.EVP_CIPHER_CTX_new()
    try:
        assert L.EVP_EncryptInit_ex(ctx, L.EVP_aes_256_ecb(), None, bytes(key), None) == 1
        L.EVP_CIPHER_CTX_set_padding(ctx, 0)
        out = ctypes.create_string_buffer(32)
        n = ctypes.c_int(0)
        assert L.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), bytes(block), 16) == 1
        return out.raw[:16]
    finally:
        L.EVP_CIPHER_CTX_free(ctx)


def gcm_encrypt(key, iv, pt):
    """(ciphertext, 16-byte tag) with a 12-byte IV and no AAD."""
    L = _lib()
    ctx = L.EVP_CIPHER_CTX_new()
    try:
        assert L.EVP_EncryptInit_ex(ctx, L.EVP_aes_256_gcm(), None, None, None) == 1
        assert L.EVP_CIPHER_CTX_ctrl(ctx, EVP_CTRL_AEAD_SET_IVLEN, len(iv), None) == 1
        assert L.EVP_EncryptInit_ex(ctx, None, None, bytes(key), bytes(iv)) == 1
        pt = bytes(pt)
        out = ctypes.create_string_buffer(len(pt) + 32)
        n = ctypes.c_int(0)
        total = 0
        if pt:
            assert L.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), pt, len(pt)) == 1
            total = n.value
        fin = ctypes.create_string_buffer(32)
        assert L.EVP_EncryptFinal_ex(ctx, fin, ctypes.byref(n)) == 1
        tag = ctypes.create_string_buffer(16)
        assert L.EVP_CIPHER_CTX_ctrl(ctx, EVP_CTRL_AEAD_GET_TAG, 16, tag) == 1
        return out.raw[:total] + fin.raw[:n.value], tag.raw
    finally:
        L.EVP_CIPHER_CTX_free(ctx)


def gcm_decrypt(key, iv, ct, tag):
    """Plaintext or None if the tag does not verify."""
    L = _lib()
    ctx = L.EVP_CIPHER_CTX_new()
    try:
        assert L.EVP_DecryptInit_ex(ctx, L.EVP_aes_256_gcm(), None, None, None) == 1
        assert L.EVP_CIPHER_CTX_ctrl(ctx, EVP_CTRL_AEAD_SET_IVLEN, len(iv), None) == 1
        assert L.EVP_DecryptInit_ex(ctx, None, None, bytes(key), bytes(iv)) == 1
        ct = bytes(ct)
        out = ctypes.create_string_buffer(len(ct) + 32)
        n = ctypes.c_int(0)
        total = 0
        if ct:
            assert L.EVP_DecryptUpdate(ctx, out, ctypes.byref(n), ct, len(ct)) == 1
            total = n.value
        tbuf = ctypes.create_string_buffer(bytes(tag), 16)
        assert L.EVP_CIPHER_CTX_ctrl(ctx, EVP_CTRL_AEAD_SET_TAG, 16, tbuf) == 1
        fin = ctypes.create_string_buffer(32)
        ok = L.EVP_DecryptFinal_ex(ctx, fin, ctypes.byref(n))
        return out.raw[:total] if ok == 1 else None
    finally:
        L.EVP_CIPHER_CTX_free(ctx)
