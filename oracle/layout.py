"""Packed 2-bit cache layouts and the bits-per-element accounting of Tab. 3.

The paper stores the cache as packed 2-bit codes plus fp16 metadata (abstract,
Sec. 3.3 "FP16 minimum and scale metadata over 32-token groups"). The byte
placement of the codes (the pack map) is this implementation's choice and is
part of its ABI; it is written out here from its definition.

Key codes, per (sequence, KV head): ``u8[cap][32]`` -- token i, channel c sits in
byte 32 i + 4 (c >> 4) + 2 (c & 1) + ((c >> 3) & 1) at bits 2 ((c >> 1) & 3) .. +1.
Read as little-endian 32-bit words, word t of a token holds channels 16 t .. 16 t + 15:
the even channels in its low half and the odd channels in its high half, two bits each
in channel order, so masking a word with 3 * 0x00010001 << 2 j leaves the codes of the
channel pair (16 t + 2 j, 16 t + 2 j + 1) in the two 16-bit halves.

Value codes, per (sequence, KV head): ``u8[cap / 32][1024]``, one 1024-byte
block per 32-token window. Inside a block, the code of window token t and
channel c sits in byte

    16 * ((c & 15) + 16 * ((t >> 2) & 3)) + 8 * (t >> 4) + (c >> 4)

at bits 2 (t & 3) .. 2 (t & 3) + 1, i.e. every byte holds one channel of four
consecutive tokens.

Metadata: fp16 key minimum and step ``[cap / 32][d]``, fp16 key and value norms
``[cap]``, modality ids ``u8[cap]`` per sequence.
"""

from __future__ import annotations

import numpy as np

WINDOW = 32
HEAD_DIM = 128


def key_byte_index(c):
    """Byte (within a token's 32) and bit shift of key channel c."""
    c = np.asarray(c)
    return 4 * (c >> 4) + 2 * (c & 1) + ((c >> 3) & 1), 2 * ((c >> 1) & 3)


def pack_keys(codes: np.ndarray) -> np.ndarray:
    """uint8 codes [n][128] (0..3) -> packed [n][32]."""
    codes = np.asarray(codes, np.uint8)
    out = np.zeros((codes.shape[0], HEAD_DIM // 4), np.uint8)
    for c in range(HEAD_DIM):
        byte, shift = key_byte_index(c)
        out[:, byte] |= (codes[:, c] << shift).astype(np.uint8)
    return out


def unpack_keys(packed: np.ndarray) -> np.ndarray:
    p = np.asarray(packed, np.uint8)
    out = np.zeros((p.shape[0], HEAD_DIM), np.uint8)
    for c in range(HEAD_DIM):
        byte, shift = key_byte_index(c)
        out[:, c] = (p[:, byte] >> shift) & 3
    return out


def value_byte_index(t: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Byte offset inside a window block of value codes for window token t and channel c."""
    t = np.asarray(t)
    c = np.asarray(c)
    return 16 * ((c & 15) + 16 * ((t >> 2) & 3)) + 8 * (t >> 4) + (c >> 4)


def pack_values(codes: np.ndarray) -> np.ndarray:
    """uint8 codes [n][128] with n a multiple of 32 -> packed [n / 32][1024]."""
    n = codes.shape[0]
    assert n % WINDOW == 0
    t, c = np.meshgrid(np.arange(WINDOW), np.arange(HEAD_DIM), indexing="ij")
    idx = value_byte_index(t, c)
    shift = (2 * (t & 3)).astype(np.uint8)
    out = np.zeros((n // WINDOW, 1024), np.uint8)
    for w in range(n // WINDOW):
        blk = codes[w * WINDOW:(w + 1) * WINDOW].astype(np.uint8)
        np.bitwise_or.at(out[w], idx.ravel(), (blk << shift).ravel().astype(np.uint8))
    return out


def unpack_values(packed: np.ndarray) -> np.ndarray:
    """packed [n_win][1024] -> uint8 codes [n_win * 32][128]."""
    n_win = packed.shape[0]
    t, c = np.meshgrid(np.arange(WINDOW), np.arange(HEAD_DIM), indexing="ij")
    idx = value_byte_index(t, c)
    shift = (2 * (t & 3)).astype(np.uint8)
    out = np.empty((n_win * WINDOW, HEAD_DIM), np.uint8)
    for w in range(n_win):
        out[w * WINDOW:(w + 1) * WINDOW] = (packed[w][idx] >> shift) & 3
    return out


# ---------------------------------------------------------------------------------------------
# MXFP4 key metadata record, one per window: 136 bytes.
#   bytes 4 q .. 4 q + 1 (little-endian 16 bits): minimum codes of channels 4 q .. 4 q + 3, channel
#                        4 q + i in bits 4 i .. 4 i + 3 (q = 0 .. 31);
#   bytes 4 q + 2 .. 4 q + 3: the step codes of the same channels;
#   byte 128 + 2 b:      E8M0 scale of the minimum block b (channels 32 b .. 32 b + 31, b = 0 .. 3);
#   byte 129 + 2 b:      E8M0 scale of the step block b.
# ---------------------------------------------------------------------------------------------
MX_RECORD = 136


def pack_mx_meta(m_codes, s_codes, m_scale, s_scale) -> np.ndarray:
    """[n_win][128] 4-bit codes and [n_win][4] scale bytes of minimum and step -> [n_win][136]."""
    m_codes, s_codes = np.asarray(m_codes, np.uint32), np.asarray(s_codes, np.uint32)
    n = m_codes.shape[0]
    out = np.zeros((n, MX_RECORD), np.uint8)
    for q in range(HEAD_DIM // 4):
        mw = sum(m_codes[:, 4 * q + i] << (4 * i) for i in range(4))
        sw = sum(s_codes[:, 4 * q + i] << (4 * i) for i in range(4))
        out[:, 4 * q] = mw & 0xFF
        out[:, 4 * q + 1] = mw >> 8
        out[:, 4 * q + 2] = sw & 0xFF
        out[:, 4 * q + 3] = sw >> 8
    out[:, 128::2] = m_scale
    out[:, 129::2] = s_scale
    return out


def unpack_mx_meta(rec: np.ndarray):
    """[n_win][136] -> (m_codes, s_codes [n_win][128], m_scale, s_scale [n_win][4])."""
    rec = np.asarray(rec, np.uint8)
    n = rec.shape[0]
    m_codes = np.zeros((n, HEAD_DIM), np.uint8)
    s_codes = np.zeros((n, HEAD_DIM), np.uint8)
    for q in range(HEAD_DIM // 4):
        mw = rec[:, 4 * q].astype(np.uint32) | (rec[:, 4 * q + 1].astype(np.uint32) << 8)
        sw = rec[:, 4 * q + 2].astype(np.uint32) | (rec[:, 4 * q + 3].astype(np.uint32) << 8)
        for i in range(4):
            m_codes[:, 4 * q + i] = (mw >> (4 * i)) & 15
            s_codes[:, 4 * q + i] = (sw >> (4 * i)) & 15
    return m_codes, s_codes, rec[:, 128:136:2].copy(), rec[:, 129:136:2].copy()


# ---------------------------------------------------------------------------------------------
# Bits per cached element (Tab. 3, "Bits/elem." column). One element = one coordinate of one
# cached key or value; the column averages keys and values.
# ---------------------------------------------------------------------------------------------

def bits_per_element(scheme: str, d: int = HEAD_DIM, group: int = WINDOW) -> float:
    """Average storage bits per K/V element for the schemes compared in Tab. 3.

    * ``turboquant_k2v2``: 2-bit codes + one fp16 norm per d-vector, for keys and values;
    * ``turboquant_k3v2``: 3-bit keys, 2-bit values, fp16 norms;
    * ``ours_fp16_meta``: values as TurboQuant K2V2; keys add an fp16 minimum and an fp16
      scale per (group of 32 tokens, channel);
    * ``ours_mxfp4_meta``: the key minimum and scale as 4-bit MXFP4 elements sharing one
      8-bit power-of-two scale per 32 metadata values.
    """
    norm = 16.0 / d
    if scheme == "turboquant_k2v2":
        k, v = 2 + norm, 2 + norm
    elif scheme == "turboquant_k3v2":
        k, v = 3 + norm, 2 + norm
    elif scheme == "ours_fp16_meta":
        k, v = 2 + norm + 2 * 16.0 / group, 2 + norm
    elif scheme == "ours_mxfp4_meta":
        k, v = 2 + norm + 2 * 4.0 / group + 2 * 8.0 / (32 * group), 2 + norm
    else:
        raise ValueError(scheme)
    return (k + v) / 2


def cache_bytes_per_token_head(d: int = HEAD_DIM, group: int = WINDOW, key_meta: str = "fp16") -> dict:
    """Bytes this layout stores per cached token per KV head, by field."""
    meta = 2 * 2 * d / group if key_meta == "fp16" else MX_RECORD / group
    return dict(k_codes=d // 4, v_codes=d // 4, k_norm=2, v_norm=2, k_meta=meta)
