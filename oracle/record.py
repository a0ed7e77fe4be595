"""Byte layout of one packed (sequence, head) state record.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper fixes the content of a stored row (Sec. 3, Levels and storage: a
width, an FP16 scale and b-bit codes per element, rows addressed through
prefix sums of the widths) and the log-uniform coding of decay rates (Sec. 3,
Decay-gate quantization); the byte layout below is this implementation's:

    0               u32 tokens seen (0 = fresh state, EMA not started)
    4               u32 reserved (0) x 3
    16              widths, 4 bits per row: b - 1, row i in byte i/2,
                    low nibble for even i
    16 + dk/2       scale   FP16 [dk]   (Delta, or mean |x| for one-bit rows)
    ... + 2 dk      zdec    u16  [dk]   log-uniform code of the rate s_hat
    ... + 2 dk      rerase  FP16 [dk]   erase rate r
    codes_off       u32 words [WC][dv]  (codes_off = meta end rounded to 256)

Codes are stored per column: column j is one bit stream holding, for rows
i = 0..dk-1 in order, the b_i-bit two's complement code of element (i, j),
least significant bit first.  Row i therefore starts at bit P_i = sum_{i'<i}
b_i' of every column (the prefix sum of widths).  Bit p of column j is bit
(p mod 32) of word [p div 32][j].  WC = ceil(dk * b_max / 32) is the capacity;
only the first ceil(sum_i b_i / 32) words of each column are meaningful and
their bits past sum_i b_i are zero.  One-bit rows store 1 for a negative
value.  The all-zero slot is the zero state.

Head units (one width per head, FP16 scales per block of 32 rows of one
column; Sec. 3, Allocation units):

    0               u32 tokens seen
    4               u32 width b of the head (0 in the zero state)
    8               u32 reserved (0) x 2
    16              zdec    u16  [dk]
    16 + 2 dk       rerase  FP16 [dk]
    16 + 4 dk       scale   FP16 [dk/32][dv]  (group: rows 32k..32k+31 of column j)
    codes_off       u32 words [WC][dv] as above with every b_i = b, so row i
                    starts at bit i b

The unquantised ("32-bit") mode stores the float32 state row-major, nothing
else.
"""
import numpy as np

HEADER = 16


def _up(x, a):
    return (x + a - 1) // a * a


def layout(dk, dv, b_max):
    w_off = HEADER
    sc_off = w_off + dk // 2
    z_off = sc_off + 2 * dk
    r_off = z_off + 2 * dk
    meta_end = r_off + 2 * dk
    codes_off = _up(meta_end, 256)
    wc = (dk * b_max + 31) // 32
    slot = _up(codes_off + wc * dv * 4, 256)
    return dict(w_off=w_off, sc_off=sc_off, z_off=z_off, r_off=r_off,
                meta_end=meta_end, codes_off=codes_off, wc=wc, slot=slot)


def record_bytes(dk, dv, b_max):
    return layout(dk, dv, b_max)["slot"]


def layout_heads(dk, dv, b_max):
    z_off = HEADER
    r_off = z_off + 2 * dk
    bs_off = r_off + 2 * dk
    meta_end = bs_off + (dk // 32) * dv * 2
    codes_off = _up(meta_end, 256)
    wc = (dk * b_max + 31) // 32
    slot = _up(codes_off + wc * dv * 4, 256)
    return dict(z_off=z_off, r_off=r_off, bs_off=bs_off, meta_end=meta_end,
                codes_off=codes_off, wc=wc, slot=slot)


def record_bytes_heads(dk, dv, b_max):
    return layout_heads(dk, dv, b_max)["slot"]


def _pack_columns(codes, widths, wc, dv):
    words = np.zeros((wc, dv), np.uint64)
    codes = np.asarray(codes, np.int64)
    widths = np.asarray(widths, np.int64)
    P = np.concatenate([[0], np.cumsum(widths)[:-1]])
    for i in range(len(widths)):
        b = int(widths[i])
        field = codes[i] & ((1 << b) - 1)
        for t in range(b):
            pos = P[i] + t
            bit = ((field >> t) & 1).astype(np.uint64)
            words[pos // 32] += bit << np.uint64(pos % 32)
    return words.astype(np.uint32)


def _unpack_columns(words, widths, dv):
    words = np.asarray(words, np.uint32).astype(np.int64)
    widths = np.asarray(widths, np.int64)
    P = np.concatenate([[0], np.cumsum(widths)[:-1]])
    codes = np.zeros((len(widths), dv), np.int64)
    for i in range(len(widths)):
        b = int(widths[i])
        field = np.zeros(dv, np.int64)
        for t in range(b):
            pos = P[i] + t
            field |= ((words[pos // 32] >> (pos % 32)) & 1) << t
        if b >= 2:
            field = np.where(field >= (1 << (b - 1)), field - (1 << b), field)
        codes[i] = field
    return codes


def pack_heads(ntok, width, scale, z, r16, codes, dk, dv, b_max):
    """Fields of one head unit -> uint8 record of record_bytes_heads."""
    L = layout_heads(dk, dv, b_max)
    buf = np.zeros(L["slot"], np.uint8)
    buf[0:4] = np.frombuffer(np.uint32(ntok).tobytes(), np.uint8)
    buf[4:8] = np.frombuffer(np.uint32(width).tobytes(), np.uint8)
    buf[L["z_off"]:L["z_off"] + 2 * dk] = np.frombuffer(np.asarray(z, np.uint16).tobytes(), np.uint8)
    buf[L["r_off"]:L["r_off"] + 2 * dk] = np.frombuffer(
        np.asarray(r16, np.float16).tobytes(), np.uint8)
    nb = (dk // 32) * dv * 2
    buf[L["bs_off"]:L["bs_off"] + nb] = np.frombuffer(
        np.asarray(scale, np.float16).reshape(-1).tobytes(), np.uint8)
    if width > 0:
        words = _pack_columns(codes, np.full(dk, width), L["wc"], dv)
        co = L["codes_off"]
        buf[co:co + L["wc"] * dv * 4] = np.frombuffer(words.tobytes(), np.uint8)
    return buf


def unpack_heads(buf, dk, dv, b_max):
    """uint8 head-unit record -> dict of fields (width 0: zero state)."""
    L = layout_heads(dk, dv, b_max)
    buf = np.asarray(buf, np.uint8)
    ntok = int(np.frombuffer(buf[0:4].tobytes(), np.uint32)[0])
    width = int(np.frombuffer(buf[4:8].tobytes(), np.uint32)[0])
    z = np.frombuffer(buf[L["z_off"]:L["z_off"] + 2 * dk].tobytes(), np.uint16).copy()
    r16 = np.frombuffer(buf[L["r_off"]:L["r_off"] + 2 * dk].tobytes(), np.float16).copy()
    nb = (dk // 32) * dv * 2
    scale = np.frombuffer(buf[L["bs_off"]:L["bs_off"] + nb].tobytes(),
                          np.float16).copy().reshape(dk // 32, dv)
    co = L["codes_off"]
    words = np.frombuffer(buf[co:co + L["wc"] * dv * 4].tobytes(), np.uint32).reshape(L["wc"], dv)
    codes = (_unpack_columns(words, np.full(dk, width), dv) if width > 0
             else np.zeros((dk, dv), np.int64))
    return dict(ntok=ntok, width=width, bscale=scale, z=z, r16=r16, codes=codes)


def meaningful_heads(buf, dk, dv, b_max):
    """Bytes of a head-unit record that carry information."""
    L = layout_heads(dk, dv, b_max)
    buf = np.asarray(buf, np.uint8)
    width = int(np.frombuffer(buf[4:8].tobytes(), np.uint32)[0])
    nw = (dk * width + 31) // 32
    return np.concatenate([buf[:L["meta_end"]], buf[L["codes_off"]:L["codes_off"] + nw * dv * 4]])


def stored_bits_heads(mean_bits, dk, dv):
    """Bits per element of the head-unit layout: payload + FP16 block scale
    (0.5) + 16-bit rate code and FP16 erase rate per row + the 32-bit width."""
    return mean_bits + 16 / 32 + (16 + 16) / dv + 32 / (dk * dv)


def state32_bytes(dk, dv):
    return dk * dv * 4


def used_words(widths):
    return (int(np.sum(widths)) + 31) // 32


def pack(ntok, widths, scale, z, r16, codes, dk, dv, b_max):
    """Fields of one head -> uint8 record of record_bytes(dk, dv, b_max)."""
    L = layout(dk, dv, b_max)
    buf = np.zeros(L["slot"], np.uint8)
    buf[0:4] = np.frombuffer(np.uint32(ntok).tobytes(), np.uint8)
    widths = np.asarray(widths, np.int64)
    nib = (widths - 1).astype(np.uint8)
    buf[L["w_off"]:L["w_off"] + dk // 2] = nib[0::2] | (nib[1::2] << 4)
    buf[L["sc_off"]:L["sc_off"] + 2 * dk] = np.frombuffer(
        np.asarray(scale, np.float16).tobytes(), np.uint8)
    buf[L["z_off"]:L["z_off"] + 2 * dk] = np.frombuffer(
        np.asarray(z, np.uint16).tobytes(), np.uint8)
    buf[L["r_off"]:L["r_off"] + 2 * dk] = np.frombuffer(
        np.asarray(r16, np.float16).tobytes(), np.uint8)
    words = np.zeros((L["wc"], dv), np.uint64)
    codes = np.asarray(codes, np.int64)
    P = np.concatenate([[0], np.cumsum(widths)[:-1]])
    for i in range(dk):
        b = int(widths[i])
        field = codes[i] & ((1 << b) - 1)
        for t in range(b):
            pos = P[i] + t
            bit = ((field >> t) & 1).astype(np.uint64)
            words[pos // 32] += bit << np.uint64(pos % 32)
    co = L["codes_off"]
    buf[co:co + L["wc"] * dv * 4] = np.frombuffer(words.astype(np.uint32).tobytes(), np.uint8)
    return buf


def unpack(buf, dk, dv, b_max):
    """uint8 record -> dict of fields (codes signed; one-bit rows 0/1)."""
    L = layout(dk, dv, b_max)
    buf = np.asarray(buf, np.uint8)
    ntok = int(np.frombuffer(buf[0:4].tobytes(), np.uint32)[0])
    nb = buf[L["w_off"]:L["w_off"] + dk // 2]
    widths = np.empty(dk, np.int64)
    widths[0::2] = (nb & 15).astype(np.int64) + 1
    widths[1::2] = (nb >> 4).astype(np.int64) + 1
    scale = np.frombuffer(buf[L["sc_off"]:L["sc_off"] + 2 * dk].tobytes(), np.float16).copy()
    z = np.frombuffer(buf[L["z_off"]:L["z_off"] + 2 * dk].tobytes(), np.uint16).copy()
    r16 = np.frombuffer(buf[L["r_off"]:L["r_off"] + 2 * dk].tobytes(), np.float16).copy()
    co = L["codes_off"]
    words = np.frombuffer(buf[co:co + L["wc"] * dv * 4].tobytes(), np.uint32).reshape(L["wc"], dv)
    words = words.astype(np.int64)
    P = np.concatenate([[0], np.cumsum(widths)[:-1]])
    codes = np.zeros((dk, dv), np.int64)
    for i in range(dk):
        b = int(widths[i])
        field = np.zeros(dv, np.int64)
        for t in range(b):
            pos = P[i] + t
            field |= ((words[pos // 32] >> (pos % 32)) & 1) << t
        if b >= 2:
            field = np.where(field >= (1 << (b - 1)), field - (1 << b), field)
        codes[i] = field
    return dict(ntok=ntok, widths=widths, scale=scale, z=z, r16=r16, codes=codes)


def meaningful(buf, dk, dv, b_max):
    """Bytes of a record that carry information (header, metadata, used words)."""
    L = layout(dk, dv, b_max)
    f = unpack(buf, dk, dv, b_max)
    nw = used_words(f["widths"])
    buf = np.asarray(buf, np.uint8)
    return np.concatenate([buf[:L["meta_end"]],
                           buf[L["codes_off"]:L["codes_off"] + nw * dv * 4]])


def accounting(mean_bits, dv, width_bits=3, block_scale=False):
    """Paper-accounted bits per element: payload + FP16 scale + width map
    (Sec. 3: 19/d_v with 3-bit widths, 20/d_v with 4-bit widths; block scales
    add 0.5)."""
    extra = 0.5 if block_scale else (16 + width_bits) / dv
    return mean_bits + extra


def stored_bits(mean_bits, dv):
    """Bits per element this layout stores: payload + width nibble + FP16
    scale + 16-bit rate code + FP16 erase rate."""
    return mean_bits + (4 + 16 + 16 + 16) / dv
