"""C3SIG-1 written out a third time, in plain Python integers, from its
specification alone.  Test infrastructure: it imports neither the oracle nor
the library, and every constant below is restated from the specification.

Sec. 5.2 asks for a deterministic, position-sensitive 64-bit hash H_w over a
tensor's dtype, shape and bytes and gives no construction.  C3SIG-1 is this
implementation's construction, applied per chunk of each tensor:

1. Words.  n = the chunk's byte length, D = 4 * ceil(n / 16); m[j] is the
   little-endian 32-bit word of bytes 4j .. 4j+3, bytes at or past n are 0.
2. Keys.  K[i], i = 0 .. 257, is the low half of the i-th output of
   SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) seeded with
   0x43335349472D3101.
3. NH fold (Black et al., UMAC, CRYPTO 1999, with a second Toeplitz row).
   For each even p < D, with q = p mod 256 and
   beta = floor(p / 256) * 0x9E3779B9 mod 2^32:
       A += (m[p] + K[q] + beta) * (m[p+1] + K[q+1] + beta)
       B += (m[p] + K[q+2] + beta) * (m[p+1] + K[q+3] + beta)
   every factor taken mod 2^32, both sums mod 2^64.
4. Finalize with MurmurHash3's fmix64 (Appleby):
       h = fmix64(0x4333534947310001 ^ (dtype << 32) ^ ndim)
       h = fmix64(h ^ dim)            for each dim of the tensor's shape
       h = fmix64(h ^ k)              k = chunk index within the tensor
       h = fmix64(h ^ n); h = fmix64(h ^ A); h = fmix64(h ^ B)
   and the chunk signature is h.

The per-tensor signature (one value per tensor, the paper's granularity) is
fmix64(0x4333534947540001 ^ S) with S the sum mod 2^64 of the tensor's chunk
signatures.  Chunk plan: a tensor of nb bytes has ceil(nb / chunk_bytes)
chunks, the last possibly partial; an empty tensor has one empty chunk.
"""
M32 = (1 << 32) - 1
M64 = (1 << 64) - 1
KEY_SEED = 0x43335349472D3101
TAG_CHUNK = 0x4333534947310001
TAG_TENSOR = 0x4333534947540001
BETA_STEP = 0x9E3779B9
ELEM_SIZE = {0: 4, 1: 2, 2: 2, 3: 1}     # F32, BF16, F16, RAW


def splitmix64(seed: int, n: int):
    """First n outputs: the state advances by the golden gamma, each output
    is the advanced state passed through the two xor-shift-multiply rounds
    and a final xor-shift."""
    out, s = [], seed & M64
    for _ in range(n):
        s = (s + 0x9E3779B97F4A7C15) & M64
        z = s
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
        out.append(z ^ (z >> 31))
    return out


def fmix64(k: int) -> int:
    k &= M64
    k ^= k >> 33
    k = (k * 0xFF51AFD7ED558CCD) & M64
    k ^= k >> 33
    k = (k * 0xC4CEB9FE1A85EC53) & M64
    k ^= k >> 33
    return k


KEYS = [v & M32 for v in splitmix64(KEY_SEED, 258)]


def nh(data: bytes):
    n = len(data)
    D = 4 * ((n + 15) // 16)
    padded = bytes(data) + bytes(4 * D - n)
    m = [int.from_bytes(padded[4 * j:4 * j + 4], "little") for j in range(D)]
    A = B = 0
    for p in range(0, D, 2):
        q = p % 256
        beta = (p // 256) * BETA_STEP & M32
        A += ((m[p] + KEYS[q] + beta) & M32) * ((m[p + 1] + KEYS[q + 1] + beta) & M32)
        B += ((m[p] + KEYS[q + 2] + beta) & M32) * ((m[p + 1] + KEYS[q + 3] + beta) & M32)
    return A & M64, B & M64


def chunk_signature(data: bytes, dtype: int, shape, k: int):
    """(A, B, sig) of one chunk: its bytes, the tensor's dtype code and shape,
    and its index k within the tensor."""
    A, B = nh(data)
    h = fmix64(TAG_CHUNK ^ (dtype << 32) ^ len(shape))
    for d in shape:
        h = fmix64(h ^ (d & M64))
    for v in (k, len(data), A, B):
        h = fmix64(h ^ v)
    return A, B, h


def tensor_nbytes(dtype: int, shape) -> int:
    n = ELEM_SIZE[dtype]
    for d in shape:
        n *= d
    return n


def chunks(tensor: bytes, chunk_bytes: int):
    """The byte slices of the chunk plan of one tensor."""
    nb = len(tensor)
    if nb == 0:
        return [b""]
    return [tensor[o:o + chunk_bytes] for o in range(0, nb, chunk_bytes)]


def tensor_signature(tensor: bytes, dtype: int, shape, chunk_bytes: int) -> int:
    s = 0
    for k, c in enumerate(chunks(tensor, chunk_bytes)):
        s = (s + chunk_signature(c, dtype, shape, k)[2]) & M64
    return fmix64(TAG_TENSOR ^ s)
