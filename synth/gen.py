"""Deterministic generators for the synthetic search-round inputs.

Every array comes from its own numpy PCG64 stream keyed by
``SeedSequence(seed, spawn_key=(cfg_id, variant, stream[, batch]))``:

====  ==========================  =========
 id   stream                      per batch
====  ==========================  =========
  1   statement counts            yes
  2   feature category            yes
  3   feature magnitude           yes
  4   split features
  5   threshold quantile q
  6   default (missing) direction
  7   leaf values
  8   threshold calibration rows
  9   policy states               yes
 10   policy weights
 11   policy biases
 12   track scores C(s)           yes
 13   track score changes         yes
 14   track critic values         yes
 15   measured-run noise          yes
 16   cut-point calibration rows
====  ==========================  =========

Nothing here computes a score, an activation or a ranking; both the oracle and the HIP path
consume these arrays as they are.
"""
from __future__ import annotations

import hashlib

import numpy as np

from .configs import RoundConfig

S_COUNTS, S_FCAT, S_FMAG, S_SPLITF, S_THRQ, S_DEFDIR, S_LEAF, S_CALIB, S_STATES, S_W, S_B = range(1, 12)
S_TRACK_C, S_TRACK_DC, S_TRACK_V = 12, 13, 14
S_MEAS_NOISE, S_MEAS_CUTS = 15, 16
_BATCH_STREAMS = {S_COUNTS, S_FCAT, S_FMAG, S_STATES, S_TRACK_C, S_TRACK_DC, S_TRACK_V, S_MEAS_NOISE}


def _rng(cfg: RoundConfig, stream: int, batch: int = 0) -> np.random.Generator:
    key = (cfg.cfg_id, cfg.variant, stream) + ((batch,) if stream in _BATCH_STREAMS else ())
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed, spawn_key=key)))


# ---------------------------------------------------------------------------------------------
# bf16 storage helpers (inputs are handed over as raw bf16 bit patterns)
# ---------------------------------------------------------------------------------------------
def bf16_bits_from_f32(x) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even) and return the 16-bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    r[np.isnan(x)] = 0x7FC0
    return r


def f32_from_bf16_bits(bits) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------------------------
# candidate programs: statement counts and per-statement features
# ---------------------------------------------------------------------------------------------
def gen_prog_ptr(cfg: RoundConfig, batch: int = 0) -> np.ndarray:
    """CSR row pointer [n_prog+1] (int32): program p owns statement rows [ptr[p], ptr[p+1])."""
    counts = _rng(cfg, S_COUNTS, batch).integers(1, cfg.s_max, size=cfg.n_prog, endpoint=True)
    ptr = np.zeros(cfg.n_prog + 1, dtype=np.int64)
    np.cumsum(counts, out=ptr[1:])
    assert ptr[-1] < 2**31
    return ptr.astype(np.int32)


def _draw_values(cat_u: np.ndarray, mag_u: np.ndarray, cfg: RoundConfig) -> np.ndarray:
    """Categorical draw per element: NaN w.p. p_nan, 0.0 w.p. p_zero, else fp32(10**U[lo,hi))."""
    out = np.power(10.0, cfg.lu_lo_exp + (cfg.lu_hi_exp - cfg.lu_lo_exp) * mag_u).astype(np.float32)
    out[cat_u < cfg.p_nan + cfg.p_zero] = 0.0
    if cfg.p_nan > 0:
        out[cat_u < cfg.p_nan] = np.nan
    return out


def gen_features(cfg: RoundConfig, n_rows: int, batch: int = 0, ld: int | None = None) -> np.ndarray:
    """Feature matrix in structure-of-arrays layout ``[n_features][ld]`` (fp32, ld >= n_rows).

    Columns past ``n_rows`` (padding) hold NaN so that a reader that strays into them shows up.
    Draw order is feature-major: feature f's row of values is drawn before feature f+1's.
    """
    ld = n_rows if ld is None else ld
    assert ld >= n_rows
    X = np.full((cfg.n_features, ld), np.nan, dtype=np.float32)
    rc, rm = _rng(cfg, S_FCAT, batch), _rng(cfg, S_FMAG, batch)
    for f in range(cfg.n_features):
        X[f, :n_rows] = _draw_values(rc.random(n_rows), rm.random(n_rows), cfg)
    return X


# ---------------------------------------------------------------------------------------------
# the GBDT cost model
# ---------------------------------------------------------------------------------------------
def gen_ensemble(cfg: RoundConfig) -> dict:
    """A GBDT of ``n_trees`` complete trees of ``depth`` split levels, in explicit node arrays.

    Tree t occupies global node ids [t*M, (t+1)*M) with M = 2**(depth+1) - 1, numbered breadth
    first: node i is internal iff i < 2**depth - 1, with children 2i+1 (left) and 2i+2 (right).
    Internal nodes carry a split feature ~U{0..F-1}, a threshold taken at a random quantile q~U[0,1)
    of that feature's calibration sample (non-missing values, sorted), and a default direction for
    missing values ~Bernoulli(0.5).  Leaves carry fp32(N(0, leaf_sigma)), or k/4096 with
    k~U{-64..64} in the exact variant.
    """
    T, D, F = cfg.n_trees, cfg.depth, cfg.n_features
    n_int, n_leaf = 2**D - 1, 2**D
    M = n_int + n_leaf
    # calibration sample, same distribution as the features
    rcal = _rng(cfg, S_CALIB)
    calib = _draw_values(rcal.random((F, cfg.n_calib)), rcal.random((F, cfg.n_calib)), cfg)
    sorted_calib = []
    for f in range(F):
        v = calib[f][~np.isnan(calib[f])]
        v.sort()
        assert v.size > 0
        sorted_calib.append(v)

    split_f = _rng(cfg, S_SPLITF).integers(0, F, size=(T, n_int))
    q = _rng(cfg, S_THRQ).random((T, n_int))
    dleft = (_rng(cfg, S_DEFDIR).random((T, n_int)) < 0.5).astype(np.uint8)
    rl = _rng(cfg, S_LEAF)
    if cfg.exact:
        leaves = (rl.integers(-64, 64, size=(T, n_leaf), endpoint=True) / 4096.0).astype(np.float32)
    else:
        leaves = rl.normal(0.0, cfg.leaf_sigma, size=(T, n_leaf)).astype(np.float32)

    thr = np.empty((T, n_int), dtype=np.float32)
    for f in range(F):
        sel = split_f == f
        sc = sorted_calib[f]
        thr[sel] = sc[(q[sel] * sc.size).astype(np.int64)]

    feature = np.full((T, M), -1, dtype=np.int32)
    threshold = np.zeros((T, M), dtype=np.float32)
    left = np.full((T, M), -1, dtype=np.int32)
    right = np.full((T, M), -1, dtype=np.int32)
    default_left = np.zeros((T, M), dtype=np.uint8)
    leaf_value = np.zeros((T, M), dtype=np.float32)
    base = (np.arange(T, dtype=np.int64) * M)[:, None]
    idx = np.arange(n_int)
    feature[:, :n_int] = split_f
    threshold[:, :n_int] = thr
    left[:, :n_int] = (base + 2 * idx + 1)
    right[:, :n_int] = (base + 2 * idx + 2)
    default_left[:, :n_int] = dleft
    leaf_value[:, n_int:] = leaves
    return dict(
        n_trees=T, n_features=F, max_depth=D,
        root=(np.arange(T, dtype=np.int64) * M).astype(np.int32),
        feature=feature.ravel(), threshold=threshold.ravel(),
        left=left.ravel(), right=right.ravel(),
        default_left=default_left.ravel(), leaf_value=leaf_value.ravel(),
        base_score=0.0,
    )


# ---------------------------------------------------------------------------------------------
# actor/critic weights and states
# ---------------------------------------------------------------------------------------------
def _store(w: np.ndarray, dtype: str) -> np.ndarray:
    w = np.ascontiguousarray(w, dtype=np.float32)
    return bf16_bits_from_f32(w) if dtype == "bf16" else w


def gen_policy(cfg: RoundConfig) -> dict:
    """Shared trunk s -> h1 -> h2 (ReLU) with an actor head h2 -> a and a value head h2 -> 1.

    Weights are ``[out][in]`` row-major, Xavier-uniform (gain 1), stored as fp32 or as bf16 bit
    patterns (round to nearest even); biases are fp32 U(-1/sqrt(fan_in), 1/sqrt(fan_in)).  The
    exact variant uses rows of at most 4 non-zeros of +-1 and integer biases in {-1, 0, 1}.
    """
    S, H1, H2, A = cfg.pol_s, cfg.pol_h1, cfg.pol_h2, cfg.pol_a
    shapes = [("w1", H1, S), ("w2", H2, H1), ("wa", A, H2), ("wv", 1, H2)]
    rw, rb = _rng(cfg, S_W), _rng(cfg, S_B)
    out = dict(dtype=cfg.pol_dtype, s=S, h1=H1, h2=H2, a=A)
    for name, fo, fi in shapes:
        if cfg.exact:
            w = np.zeros((fo, fi), dtype=np.float32)
            for r in range(fo):
                nnz = int(rw.integers(0, 4, endpoint=True))
                pos = rw.choice(fi, size=nnz, replace=False)
                w[r, pos] = rw.choice(np.array([-1.0, 1.0], dtype=np.float32), size=nnz)
        else:
            a = np.sqrt(6.0 / (fi + fo))
            w = rw.uniform(-a, a, size=(fo, fi)).astype(np.float32)
        out[name] = _store(w, cfg.pol_dtype)
    for name, fo, fi in [("b1", H1, S), ("b2", H2, H1), ("ba", A, H2), ("bv", 1, H2)]:
        if cfg.exact:
            b = rb.integers(-1, 1, size=fo, endpoint=True).astype(np.float32)
        else:
            bound = 1.0 / np.sqrt(fi)
            b = rb.uniform(-bound, bound, size=fo).astype(np.float32)
        out[name] = b
    return out


def gen_states(cfg: RoundConfig, batch: int = 0, n: int | None = None) -> np.ndarray:
    """Policy observations ``[n][pol_s]`` row-major: fp32 N(0,1) (bf16 bits for bf16 policies);
    the exact variant draws from {-1, 0, 1}."""
    n = cfg.n_prog if n is None else n
    r = _rng(cfg, S_STATES, batch)
    if cfg.exact:
        s = r.integers(-1, 1, size=(n, cfg.pol_s), endpoint=True).astype(np.float32)
    else:
        s = r.standard_normal((n, cfg.pol_s)).astype(np.float32)
    return _store(s, cfg.pol_dtype)


def gen_track_step(cfg: RoundConfig, batch: int = 0, n: int | None = None) -> dict:
    """One modification step of n schedule tracks (fp32 arrays [n]): cost-model scores before and
    after (c_prev ~ N(0, 7^2), the spread of the standard round's program scores; c_next = c_prev
    + N(0, 1), equal to c_prev for 5 % of the tracks, the dummy action) and critic values
    v_prev, v_next ~ N(0, 1).  The exact variant draws c_prev = +-2^e (e in -2..3), changes k/8
    (|k| <= 8) and values k/16, so every reward and advantage (gamma = 0.5) is exact in fp32."""
    n = cfg.n_prog if n is None else n
    rc, rd, rv = _rng(cfg, S_TRACK_C, batch), _rng(cfg, S_TRACK_DC, batch), _rng(cfg, S_TRACK_V, batch)
    if cfg.exact:
        c0 = (rc.choice([-1.0, 1.0], n) * np.exp2(rc.integers(-2, 3, n, endpoint=True))).astype(np.float32)
        c1 = (c0 + rd.integers(-8, 8, n, endpoint=True) / 8.0).astype(np.float32)
        v = (rv.integers(-16, 16, (2, n), endpoint=True) / 16.0).astype(np.float32)
    else:
        c0 = (rc.standard_normal(n) * 7.0).astype(np.float32)
        dc = rd.standard_normal(n)
        dc[rd.random(n) < 0.05] = 0.0
        c1 = (c0 + dc).astype(np.float32)
        v = rv.standard_normal((2, n)).astype(np.float32)
    return dict(c_prev=c0, c_next=c1, v_prev=v[0].copy(), v_next=v[1].copy())


def gen_measured(cfg: RoundConfig, n_cuts: int = 254, batch: int = 0) -> dict:
    """Measured programs for a refit of the cost model: the batch's programs and statement features
    (as gen_batch: prog_ptr, features [F][n_rows]), a measured throughput per program and per-feature
    cut points.

    A statement's synthetic run time is 0.1 + log10(1 + |x3|) + 0.5 [x17 > 1] + 0.25 log10(1 + |x101|)
    (missing values count 0; feature ids taken modulo F), a program's is the sum over its statements
    times a log-normal factor exp(N(0, 0.1^2)); label = throughput / the largest throughput, and
    weight = label (Ansor weights each program's squared error by its normalised throughput).
    Cut points: per feature, the distinct values at n_cuts + 1 equally spaced ranks of a sorted
    calibration sample of non-missing values (at most n_cuts of them, strictly increasing), in
    cuts [F][n_cuts] (unused tail 0) with counts n_cuts_f [F]."""
    ptr = gen_prog_ptr(cfg, batch)
    n_rows = int(ptr[-1])
    X = gen_features(cfg, n_rows, batch)
    F = cfg.n_features
    xz = np.nan_to_num(X.astype(np.float64), nan=0.0)
    row_t = 0.1 + np.log10(1 + np.abs(xz[3 % F])) + 0.5 * (xz[17 % F] > 1) + 0.25 * np.log10(1 + np.abs(xz[101 % F]))
    prog_t = np.add.reduceat(row_t, ptr[:-1]) if n_rows else np.zeros(cfg.n_prog)
    prog_t[np.diff(ptr) == 0] = 0.1
    prog_t *= np.exp(_rng(cfg, S_MEAS_NOISE, batch).normal(0.0, 0.1, cfg.n_prog))
    thr = 1.0 / prog_t
    label = (thr / thr.max()).astype(np.float32)
    rcal = _rng(cfg, S_MEAS_CUTS)
    cal_cfg = cfg.with_(p_nan=0.0)
    calib = _draw_values(rcal.random((F, cfg.n_calib)), rcal.random((F, cfg.n_calib)), cal_cfg)
    cuts = np.zeros((F, max(n_cuts, 1)), np.float32)
    counts = np.zeros(F, np.int32)
    ranks = (np.arange(1, n_cuts + 1) * cfg.n_calib) // (n_cuts + 1)
    for f in range(F):
        v = np.unique(np.sort(calib[f])[ranks])
        counts[f] = v.size
        cuts[f, :v.size] = v
    return dict(prog_ptr=ptr, n_rows=n_rows, features=X, label=label, weight=label.copy(), cuts=cuts,
                n_cuts=counts)


def gen_batch(cfg: RoundConfig, batch: int = 0, ld_pad: int = 0) -> dict:
    """All per-batch inputs of one round: prog_ptr, features (SoA) and states."""
    ptr = gen_prog_ptr(cfg, batch)
    n_rows = int(ptr[-1])
    X = gen_features(cfg, n_rows, batch, ld=n_rows + ld_pad)
    return dict(prog_ptr=ptr, n_rows=n_rows, features=X, ld=X.shape[1],
                states=gen_states(cfg, batch))


def digest(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()
