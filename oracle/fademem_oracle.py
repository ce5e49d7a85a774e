"""Plain CPU oracle of FadeMem's per-chunk cache step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module: only the tests, the smoke check and the CPU-baseline leg of the
benchmark use it.  It shares no code, table or helper with the HIP library.

What it computes (FadeMem, arXiv 2606.10671):

* Memory entries and insertion -- Sec. 3.3 "Memory entries and insertion":
  an ordered memory of at most M entries m_i = (K_i, V_i, mu_i, s_i); a new
  block enters as (K_t, V_t, t, 1).
* Distance-aware scheduling -- Sec. 3.3 "Distance-aware scheduling" and
  Algorithm S1: d_i = t - mu_i, u(d) = d**beta, the adjacent pair with the
  smallest |u(d_{i+1}) - u(d_i)| is chosen; the pair holding the newest
  entry is not eligible (Sec. 3.3 "Boundary and positional handling",
  Algorithm S1).
* Consolidation operator -- Sec. 3.3 "Consolidation operator": spans add,
  mu is the span-weighted mean, K and V are square-root-span weighted
  averages.  The first-frame anchor keeps its K, V and position when its
  pair is chosen (Algorithm S1, supplementary Sec. S1).  The ablation of
  Sec. 4.3 ("Memory consolidation operator", Table 4) swaps the K, V rule
  for an unweighted average, a representative selection ("Select Nearest")
  or elementwise max pooling; the metadata rule is the same for all.
* Attention -- Sec. 3.1: the chunk's queries attend over the exposed cache
  [memory entries in order || current chunk].  This is textbook softmax
  attention, written out in fp64.
* Temporal RoPE handling -- Sec. 3.3 "Boundary and positional handling":
  memory keys are kept without their temporal rotary phase and re-indexed
  within a bounded temporal range at attention time.  The rotation of one
  pair of dimensions by an angle is the plane rotation of rotary position
  embeddings; which index each retained entry gets is a reading (below).

Readings where the paper is silent (each is listed with its reason in the
design notes of the repository):

* positions are 0-indexed integers given by the caller; the anchor's
  position is the first inserted position (Algorithm S1 sets it to 0, which
  is that position under 0-indexing);
* mu is held exactly as the rational pos_sum / span with integer pos_sum;
  d_i is evaluated as (t*s_i - pos_sum_i) / s_i with one rounding in fp64;
* u(d) and the gaps are fp64; ties (relative 1e-9) go to the lowest index;
* t in d_i = t - mu_i is the newest entry's position;
* merged K, V are evaluated in fp64 exactly as the paper writes them
  (two products and one sum, each rounded to fp64) and rounded once to the
  storage type (fp32, or bf16 with round-to-nearest-even);
* a chunk of F frames runs F insert+consolidate updates in frame order,
  after the chunk's attention call;
* "Select Nearest" keeps the newer entry's K, V (the entry nearer to the
  present, whose distance the schedule measures); max pooling takes, per
  element, the newer entry's value when it is strictly greater, else the
  older one's (so equal values, including -0 and +0, keep the older bits);
* temporal RoPE: the first P interleaved pairs (2k, 2k+1) of a head carry
  the temporal phase, pair k at frequency theta**(-k/P) (the layout of a
  video model's temporal rotary axis); memory entry i (0 = oldest) is
  exposed at temporal index i and the current chunk's frame f at n + f
  (n = entries held).  Parity unpinned as to the paper: the paper does not
  state the mapping.  The rotation itself is pinned (complex
  multiplication, composition, relative-position invariance).

Parity status: every function here is pinned by tests under tests/ (see
tests/test_oracle_*.py) except where a docstring says "parity unpinned".
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

TIE_RTOL = 1e-9  # relative tolerance under which two gaps count as tied
OPERATORS = ("sqrt_span", "average", "select_nearest", "max")  # Sec. 3.3 default, then Table 4


# ---------------------------------------------------------------------------
# Storage rounding (the paper computes in BF16: Sec. 4.1 and supplementary
# Sec. S4).  The oracle rounds by definition: to the nearest multiple of the
# format's spacing, ties to even.
# ---------------------------------------------------------------------------

def round_to_bf16(x) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16 number, ties to even.

    bfloat16 has 8 significant bits and fp32's exponent range (normals from
    2**-126, subnormal spacing 2**-133).  For |x| in [2**e, 2**(e+1)) the
    spacing of bfloat16 numbers is 2**(e-7); dividing by a power of two is
    exact, so np.round (half to even) on the scaled value performs the
    rounding exactly.  Values at or beyond the overflow midpoint become inf.
    Returns float32 arrays (every bfloat16 number is an fp32 number).
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(np.abs(x))          # |x| = m * 2**e, m in [0.5, 1)
    e = np.maximum(e - 1, -126)         # |x| in [2**e, 2**(e+1)); subnormal floor
    q = np.ldexp(np.ones_like(x), e - 7)
    r = np.round(x / q) * q
    with np.errstate(over="ignore"):
        return r.astype(np.float32)     # exact, except 2**128 -> inf


def round_to_f32(x) -> np.ndarray:
    """Round fp64 values to fp32 (IEEE round-to-nearest-even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def bf16_bits(x) -> np.ndarray:
    """uint16 bit patterns of bfloat16-representable float32 values."""
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def bf16_from_bits(b) -> np.ndarray:
    """float32 values of uint16 bfloat16 bit patterns (exact)."""
    b = np.ascontiguousarray(np.asarray(b, dtype=np.uint16))
    return (b.astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# The bounded ordered memory (Sec. 3.1, Sec. 3.3, Algorithm S1).
# ---------------------------------------------------------------------------

@dataclass
class Entry:
    """One memory entry m_i = (K_i, V_i, mu_i, s_i) (Sec. 3.3).

    mu_i is kept exactly as pos_sum / span: pos_sum is the sum of the
    positions of the blocks the entry covers, so the consolidation rule
    s_new * mu_new = s_j mu_j + s_{j+1} mu_{j+1} becomes an integer sum.
    ``first`` is the first position the entry covers.
    """
    first: int
    pos_sum: int
    span: int
    anchor: bool
    K: np.ndarray
    V: np.ndarray

    @property
    def mu(self) -> float:
        return self.pos_sum / self.span


@dataclass
class OracleCache:
    """FadeMem memory of one layer (or of several layers sharing one
    schedule: K and V may carry any leading shape, merges are elementwise).

    budget  -- M, the entry budget (Sec. 3.1); M >= 2 so that at least one
               pair stays eligible once the newest is protected.
    beta    -- exponent of u(d) = d**beta, 0 < beta <= 1 (Sec. 3.3).
    anchor  -- keep the first block as a global anchor (Sec. 3.3, S1).
    storage -- "f32" or "bf16": the type merged K, V are stored in.
    operator -- the K, V rule of a merge: "sqrt_span" (the default of
               Sec. 3.3), or one of the Table 4 ablations "average",
               "select_nearest", "max".
    """
    budget: int
    beta: float = 0.3
    anchor: bool = True
    storage: str = "f32"
    operator: str = "sqrt_span"
    entries: List[Entry] = field(default_factory=list)
    newest: Optional[int] = None
    merge_log: List[int] = field(default_factory=list)
    anchor_merges: int = 0
    weighted_merges: int = 0

    def __post_init__(self):
        if self.budget < 2:
            raise ValueError("budget must be >= 2")
        if not (0.0 < self.beta <= 1.0):
            raise ValueError("beta must satisfy 0 < beta <= 1")
        if self.storage not in ("f32", "bf16"):
            raise ValueError("storage must be 'f32' or 'bf16'")
        if self.operator not in OPERATORS:
            raise ValueError(f"operator must be one of {OPERATORS}")

    # -- storage rounding -------------------------------------------------
    def _store(self, x64: np.ndarray) -> np.ndarray:
        if self.storage == "bf16":
            return round_to_bf16(x64)
        return round_to_f32(x64)

    # -- Algorithm S1, first step: Append --------------------------------
    def insert(self, K: np.ndarray, V: np.ndarray, t: int) -> None:
        """Append the new entry (K_t, V_t, t, 1) (Sec. 3.3, Algorithm S1).

        K and V must already be representable in the storage type.  The
        first block inserted into an empty memory is the anchor when the
        anchor option is on.
        """
        t = int(t)
        if self.entries and t <= self.newest:
            raise ValueError("positions must strictly increase")
        if len(self.entries) > self.budget:
            raise ValueError("consolidate before inserting again")
        K = np.array(K, dtype=np.float32, copy=True)
        V = np.array(V, dtype=np.float32, copy=True)
        if self.storage == "bf16":
            if not (np.array_equal(round_to_bf16(K), K, equal_nan=True)
                    and np.array_equal(round_to_bf16(V), V, equal_nan=True)):
                raise ValueError("K, V are not bfloat16 values")
        is_anchor = self.anchor and not self.entries
        self.entries.append(Entry(first=t, pos_sum=t, span=1, anchor=is_anchor, K=K, V=V))
        self.newest = t

    # -- Algorithm S1, schedule -------------------------------------------
    def distances(self) -> List[float]:
        """d_i = t - mu_i for every entry, t = the newest position.

        Evaluated as (t*s_i - pos_sum_i) / s_i: an exact integer numerator
        and one correctly rounded fp64 division.
        """
        t = self.newest
        return [float(t * e.span - e.pos_sum) / float(e.span) for e in self.entries]

    def gaps(self) -> List[float]:
        """g_i = |u(d_{i+1}) - u(d_i)| for the eligible pairs (i, i+1).

        The pair that contains the newest entry (the last one) is excluded,
        so with n entries the eligible pairs are i = 0 .. n-3.
        """
        d = self.distances()
        u = [di ** self.beta for di in d]
        n = len(self.entries)
        return [abs(u[i + 1] - u[i]) for i in range(n - 2)]

    def select(self) -> int:
        """j = argmin_i g_i, ties (within TIE_RTOL relative) to the lowest i."""
        g = self.gaps()
        gm = min(g)
        for i, gi in enumerate(g):
            if gi - gm <= TIE_RTOL * gm:
                return i
        raise AssertionError("unreachable")

    @staticmethod
    def weights(s_j: int, s_j1: int) -> Tuple[float, float]:
        """w_j = sqrt(s_j) / (sqrt(s_j) + sqrt(s_{j+1})), w_{j+1} = 1 - w_j
        (Sec. 3.3 "Consolidation operator", Algorithm S1), in fp64."""
        rj = math.sqrt(s_j)
        rj1 = math.sqrt(s_j1)
        w_j = rj / (rj + rj1)
        return w_j, 1.0 - w_j

    def merge_values(self, a: Entry, b: Entry) -> Tuple[np.ndarray, np.ndarray]:
        """K, V of the merged entry under the configured operator:

        sqrt_span      -- K_new = w_j K_j + w_{j+1} K_{j+1} with the weights
                          above (Sec. 3.3), in fp64, then one rounding to the
                          storage type;
        average        -- the same with w_j = w_{j+1} = 1/2 (Table 4);
        select_nearest -- the newer entry's K, V as stored (Table 4);
        max            -- elementwise maximum of the stored values (Table 4).
        """
        if self.operator == "select_nearest":
            return b.K.copy(), b.V.copy()
        if self.operator == "max":
            return tuple(np.where(xb > xa, xb, xa) for xa, xb in ((a.K, b.K), (a.V, b.V)))
        if self.operator == "average":
            w_j, w_j1 = 0.5, 0.5
        else:
            w_j, w_j1 = self.weights(a.span, b.span)
        out = []
        for xa, xb in ((a.K, b.K), (a.V, b.V)):
            xa64 = xa.astype(np.float64)
            xb64 = xb.astype(np.float64)
            prod_a = w_j * xa64
            prod_b = w_j1 * xb64
            out.append(self._store(prod_a + prod_b))
        return out[0], out[1]

    def consolidate(self) -> Optional[int]:
        """Rest of Algorithm S1: return if |M_t| <= M, else merge the pair
        chosen by the schedule and replace it by the merged entry.  Returns
        the selected index j, or None when no merge was needed."""
        n = len(self.entries)
        if n <= self.budget:
            return None
        j = self.select()
        a, b = self.entries[j], self.entries[j + 1]
        s_new = a.span + b.span
        if a.anchor:
            # anchor pair: spans add, the anchor's K, V and position stay
            merged = Entry(first=a.first, pos_sum=a.first * s_new, span=s_new,
                           anchor=True, K=a.K, V=a.V)
            self.anchor_merges += 1
        else:
            K_new, V_new = self.merge_values(a, b)
            merged = Entry(first=a.first, pos_sum=a.pos_sum + b.pos_sum, span=s_new,
                           anchor=False, K=K_new, V=V_new)
            self.weighted_merges += 1
        self.entries[j:j + 2] = [merged]
        self.merge_log.append(j)
        return j

    def update(self, K: np.ndarray, V: np.ndarray, t: int) -> Optional[int]:
        """One full Algorithm S1 update: insert, then consolidate."""
        self.insert(K, V, t)
        return self.consolidate()

    # -- views --------------------------------------------------------------
    def state(self) -> dict:
        return {
            "count": len(self.entries),
            "first": [e.first for e in self.entries],
            "span": [e.span for e in self.entries],
            "pos_sum": [e.pos_sum for e in self.entries],
            "newest": self.newest,
        }

    def exposed_kv(self) -> Tuple[List[np.ndarray], List[np.ndarray]]:
        return [e.K for e in self.entries], [e.V for e in self.entries]


# ---------------------------------------------------------------------------
# Attention over [memory || current chunk] (Sec. 3.1; 15-slot exposure in
# Sec. 4.1).  Plain softmax attention, no mask, scale 1/sqrt(D).
# ---------------------------------------------------------------------------

def attend(Q: np.ndarray, K_mem: Sequence[np.ndarray], V_mem: Sequence[np.ndarray],
           K_cur: np.ndarray, V_cur: np.ndarray, scale: Optional[float] = None,
           q_block: int = 1024) -> Tuple[np.ndarray, np.ndarray]:
    """O_h = softmax(Q_h K_h^T * scale) V_h for every head h, in fp64.

    Q          -- [Lq][H][D]
    K_mem/V_mem-- memory entries in memory order, each [N][H][D]
    K_cur/V_cur-- current chunk, [Lc][H][D]
    Returns O [Lq][H][D] (fp64) and LSE [H][Lq] (natural log of the softmax
    denominator of the scaled scores).
    """
    Q = np.asarray(Q, dtype=np.float64)
    Lq, H, D = Q.shape
    if scale is None or scale == 0.0:
        scale = 1.0 / math.sqrt(D)
    K_all = np.concatenate([np.asarray(k, np.float64) for k in K_mem] + [np.asarray(K_cur, np.float64)], axis=0)
    V_all = np.concatenate([np.asarray(v, np.float64) for v in V_mem] + [np.asarray(V_cur, np.float64)], axis=0)
    O = np.zeros((Lq, H, D), dtype=np.float64)
    LSE = np.zeros((H, Lq), dtype=np.float64)
    for h in range(H):
        Kh = K_all[:, h, :]
        Vh = V_all[:, h, :]
        for q0 in range(0, Lq, q_block):
            Qb = Q[q0:q0 + q_block, h, :]
            S = (Qb @ Kh.T) * scale
            m = S.max(axis=1, keepdims=True)
            P = np.exp(S - m)
            denom = P.sum(axis=1, keepdims=True)
            O[q0:q0 + q_block, h, :] = (P @ Vh) / denom
            LSE[h, q0:q0 + q_block] = (m + np.log(denom))[:, 0]
    return O, LSE


# ---------------------------------------------------------------------------
# Temporal RoPE re-indexing (Sec. 3.3 "Boundary and positional handling").
# ---------------------------------------------------------------------------

def rope_angles(index: float, pairs: int, theta: float) -> np.ndarray:
    """Angle of pair k = 0..P-1 at temporal `index`: index * theta**(-k/P) (fp64)."""
    k = np.arange(pairs, dtype=np.float64)
    return float(index) * np.power(float(theta), -k / float(pairs))


def rope_rotate(X: np.ndarray, index: float, pairs: int, theta: float, storage: Optional[str] = None) -> np.ndarray:
    """Rotate pairs (2k, 2k+1), k < P, of the last axis of X by rope_angles:
    (x0, x1) -> (x0 c - x1 s, x0 s + x1 c), products and sums in fp64; the
    other dimensions are unchanged.  storage: round the result once to
    "bf16" or "f32", or keep fp64 (None)."""
    Y = np.array(X, dtype=np.float64, copy=True)
    if pairs > 0:
        a = rope_angles(index, pairs, theta)
        c, s = np.cos(a), np.sin(a)
        x0 = Y[..., 0:2 * pairs:2].copy()
        x1 = Y[..., 1:2 * pairs:2].copy()
        Y[..., 0:2 * pairs:2] = x0 * c - x1 * s
        Y[..., 1:2 * pairs:2] = x0 * s + x1 * c
    if storage == "bf16":
        return round_to_bf16(Y)
    if storage == "f32":
        return round_to_f32(Y)
    return Y


def exposed_kv_rope(cache: "OracleCache", pairs: int, theta: float) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """The memory as attention sees it with temporal RoPE handling: entry i's
    keys rotated to temporal index i (and rounded to the storage type, as the
    library's exposed copy is), values unchanged.  Parity unpinned as to the
    paper's mapping (see the module docstring)."""
    K = [rope_rotate(e.K, i, pairs, theta, cache.storage) for i, e in enumerate(cache.entries)]
    return K, [e.V for e in cache.entries]


def chunk_step(cache: OracleCache, Q: np.ndarray, K_chunk: np.ndarray, V_chunk: np.ndarray,
               frames: int, first_position: int, attend_fn=None):
    """One generated chunk: attention of the chunk's queries over
    [memory || chunk], then one insert+consolidate per frame in frame order
    (Sec. 4.1: memory updated after the final denoising step; each entry
    stores one latent frame, supplementary Sec. S4).

    K_chunk/V_chunk are [frames*N][H][D].  Returns (O, LSE, merges)."""
    K_mem, V_mem = cache.exposed_kv()
    fn = attend if attend_fn is None else attend_fn
    O, LSE = fn(Q, K_mem, V_mem, K_chunk, V_chunk)
    N = K_chunk.shape[0] // frames
    merges = []
    for f in range(frames):
        merges.append(cache.update(K_chunk[f * N:(f + 1) * N], V_chunk[f * N:(f + 1) * N],
                                   first_position + f))
    return O, LSE, merges


# ---------------------------------------------------------------------------
# Distance-dependent spectral decay (Sec. 3.2; supplementary Sec. S2): an
# orthonormal 2-D DCT-II of each channel-averaged latent frame, coefficients
# grouped by normalized radial frequency r(u, v) = sqrt((u/H)^2 + (v/W)^2),
# the Pearson correlation C_k(lag) between band k's coefficients of frame 0
# and of frame lag, averaged over clips; per band a decorrelation horizon,
# and the fit r*(t) = a t^(-b) by nonlinear least squares.
# Readings where the paper is silent: `bands` equal-width bands of r over
# [0, max r] with the DC coefficient left out; the curve is smoothed with a
# centred moving average of 5 lags (shrinking at the ends); the horizon is
# the first lag, after at least half of the curve's total decay, at which
# the smoothed curve falls by less than 5 % of its steepest one-lag fall
# (for a decay exp(-lag/tau) that is tau*ln 20, proportional to tau); a
# band's radius is the centre of its bin.
# ---------------------------------------------------------------------------

def dct2_ortho(Z) -> np.ndarray:
    """Orthonormal 2-D DCT-II over the last two axes, in fp64 (library DCT)."""
    from scipy.fft import dctn
    return dctn(np.asarray(Z, dtype=np.float64), type=2, norm="ortho", axes=(-2, -1))


def radial_band_of(H: int, W: int, bands: int) -> Tuple[np.ndarray, np.ndarray]:
    """Band index of every coefficient (u, v) as an int32 [H][W] array (-1 for
    the DC coefficient) and the bands' centre radii."""
    r = np.sqrt((np.arange(H)[:, None] / H) ** 2 + (np.arange(W)[None, :] / W) ** 2)
    r_max = r.max()
    k = np.minimum(np.floor(r / r_max * bands).astype(np.int64), bands - 1)
    k[0, 0] = -1
    centres = (np.arange(bands) + 0.5) * r_max / bands
    return k.astype(np.int32), centres


def pearson(x: np.ndarray, y: np.ndarray) -> float:
    """Pearson correlation coefficient, by its definition, in fp64."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    xm = x - x.mean()
    ym = y - y.mean()
    return float((xm @ ym) / math.sqrt((xm @ xm) * (ym @ ym)))


def band_correlations(latents, band_of: np.ndarray, bands: int, max_lag: int) -> np.ndarray:
    """C_k(lag) for k < bands, lag = 0..max_lag: per clip the Pearson
    correlation of band k's DCT coefficients of frame 0 and frame lag,
    averaged over clips.  latents: [clips][frames][H][W]."""
    L = np.asarray(latents)
    out = np.zeros((bands, max_lag + 1))
    for c in range(L.shape[0]):
        D = dct2_ortho(L[c, :max_lag + 1])
        for k in range(bands):
            sel = band_of == k
            x = D[0][sel]
            for lag in range(max_lag + 1):
                out[k, lag] += pearson(x, D[lag][sel])
    return out / L.shape[0]


def decorrelation_horizons(corr: np.ndarray, width: int = 5, drop: float = 0.05) -> np.ndarray:
    """Per band, the lag at which the smoothed curve enters its near-flat
    regime (the reading in the section comment); -1 if it never does."""
    bands, n = corr.shape
    out = np.full(bands, -1, dtype=np.int64)
    h = width // 2
    for k in range(bands):
        s = np.array([corr[k, max(0, i - h):min(n, i + h + 1)].mean() for i in range(n)])
        total = s[0] - s.min()
        steepest = (s[:-1] - s[1:]).max() if n > 1 else 0.0
        if not (total > 0 and steepest > 0):
            continue
        for lag in range(1, n - 1):
            if s[0] - s[lag] >= 0.5 * total and s[lag] - s[lag + 1] < drop * steepest:
                out[k] = lag
                break
    return out


def fit_power_law(t: np.ndarray, r: np.ndarray) -> Tuple[float, float]:
    """(a, b) of r = a * t^(-b) by nonlinear least squares (library solver)."""
    from scipy.optimize import curve_fit
    t = np.asarray(t, np.float64)
    r = np.asarray(r, np.float64)
    b0, la0 = np.polyfit(np.log(t), np.log(r), 1)
    (a, b), _ = curve_fit(lambda x, a, b: a * np.power(x, -b), t, r, p0=(math.exp(la0), -b0), maxfev=10000)
    return float(a), float(b)
