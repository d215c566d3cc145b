"""Counter-based random stream and the per-iteration pattern sampler.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper draws a pattern period ``dp`` from the searched distribution K and
then a bias ``b`` uniformly from {1..dp} in every iteration (Sec. III-D), but
names no generator. The reading used here:

* generator: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
  number generators", OOPSLA 2014), i.e. a Weyl sequence with increment
  0x9E3779B97F4A7C15 followed by the variant-13 64-bit finaliser;
* one independent stream per (seed, stream, iteration): the initial state is
  ``seed XOR ((stream << 40) | iteration)`` with stream < 2**24 and
  iteration < 2**40, so any iteration can be replayed without the ones before;
* a uniform double is ``(w >> 11) * 2**-53``;
* the period is the smallest i (1-based) whose running sum
  ``C_i = C_{i-1} + k_i`` (sequential fp64 additions, ``C_0 = 0``) exceeds the
  uniform; if rounding leaves none, the largest i with ``k_i > 0``;
* the offset ``b - 1`` is an unbiased draw from {0..dp-1} by modulo rejection:
  redraw while ``w < 2**64 mod dp``, then take ``w mod dp``.

Pure Python integers are used so that every step is exact and readable.
"""

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15
MIX_1 = 0xBF58476D1CE4E5B9
MIX_2 = 0x94D049BB133111EB

STREAM_BITS = 24
ITER_BITS = 40


def splitmix64_next(state):
    """One SplitMix64 step: returns (new_state, 64-bit output)."""
    state = (state + GOLDEN_GAMMA) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * MIX_1) & MASK64
    z = ((z ^ (z >> 27)) * MIX_2) & MASK64
    return state, z ^ (z >> 31)


class CounterStream:
    """The SplitMix64 stream of one (seed, stream, iteration) triple."""

    def __init__(self, seed, stream, iteration):
        if not (0 <= stream < (1 << STREAM_BITS)):
            raise ValueError("stream must be < 2**24")
        if not (0 <= iteration < (1 << ITER_BITS)):
            raise ValueError("iteration must be < 2**40")
        self.state = (seed & MASK64) ^ ((stream << ITER_BITS) | iteration)

    def next_u64(self):
        self.state, out = splitmix64_next(self.state)
        return out

    def next_uniform(self):
        """A double in [0, 1) with 53 random bits."""
        return (self.next_u64() >> 11) * (2.0 ** -53)

    def next_below(self, n):
        """Unbiased integer in [0, n) by modulo rejection."""
        if n <= 0:
            raise ValueError("n must be positive")
        threshold = (1 << 64) % n
        w = self.next_u64()
        while w < threshold:
            w = self.next_u64()
        return w % n


def sample_period(K, u):
    """Inverse-CDF draw of the period dp in {1..len(K)} from uniform u (Sec. III-D).

    The CDF is built by sequential fp64 additions in index order.
    """
    c = 0.0
    for i, k in enumerate(K):
        c = c + float(k)
        if u < c:
            return i + 1
    last = 0
    for i, k in enumerate(K):
        if float(k) > 0.0:
            last = i + 1
    if last == 0:
        raise ValueError("K has no positive entry")
    return last


def sample_row_pattern(K, seed, stream, iteration):
    """Draw (period, offset) for one dropout layer in one iteration (Sec. III-D).

    ``offset`` is the 0-based bias: the paper's b equals offset + 1.
    """
    g = CounterStream(seed, stream, iteration)
    period = sample_period(K, g.next_uniform())
    offset = g.next_below(period)
    return period, offset


def tile_bitmap_tdp(tiles_n, tiles_k, period, offset):
    """Kept-tile bitmap of a tile-based pattern (Sec. III-B).

    Tiles of W[N][K] are numbered row-major, t = tn * tiles_k + tk ("successive
    tiles"); tile t is kept iff t mod period == offset. Returns a list of 32-bit
    words: bit t lives in word t // 32 at position t % 32.
    """
    total = tiles_n * tiles_k
    words = [0] * ((total + 31) // 32)
    for t in range(total):
        if t % period == offset:
            words[t // 32] |= 1 << (t % 32)
    return words


def tile_bitmap_bernoulli(tiles_n, tiles_k, p, seed, stream, iteration):
    """DropConnect-style tile bitmap: tile t uses the t-th draw of the stream and
    is kept iff that uniform is >= p (keep probability 1 - p)."""
    total = tiles_n * tiles_k
    g = CounterStream(seed, stream, iteration)
    words = [0] * ((total + 31) // 32)
    for t in range(total):
        if g.next_uniform() >= p:
            words[t // 32] |= 1 << (t % 32)
    return words
