"""Seeded synthetic inputs for the sparse basis convolution.

This module only draws inputs: coordinates, event streams, features, weights
and upstream gradients.  It holds none of the convolution's arithmetic (no
neighbour test, no basis, no products), so that the CPU oracle and the HIP
path can both be fed the very same bytes without sharing any of the method.

Shapes follow the paper's workloads:
  * point clouds stand in for ModelNet40 examples (1024 surface points per
    cloud, Section 4 "Experiments"), concatenated as a ragged batch
    (Section 3.1 "Ragged Batching");
  * event streams stand in for the DVS datasets of the supplementary Table 7
    (128x128 sensors, a few hundred thousand events, cropped at 300k).

Every generator draws in float64 and casts once.  bf16 values are produced by
round-to-nearest-even from the float32 draw and handed out both as raw bit
patterns (uint16) and as the float32 numbers they denote.
"""
from __future__ import annotations

import numpy as np

ROOT_SEED = 20120117

# basis identifiers shared by both sides (just names, no arithmetic)
BASIS_MONO4 = "mono4"      # {1, ux, uy, uz} x window, M = 4
BASIS_MONO8 = "mono8"      # {1, ux, uy, uz, ux^2, uy^2, uz^2, ux*uy} x window, M = 8
BASIS_EVENT8 = "event8"    # 3x3 pixel offsets without the centre, x exp decay, M = 8
BASIS_WMONO10 = "wmono10"  # weighted convolution, all monomials up to 2nd order, M = 10
BASIS_EVENT_DECAYS = "event_decays"  # 3x3 offsets without the centre x M_v decays, M = 8 M_v

BASIS_M = {BASIS_MONO4: 4, BASIS_MONO8: 8, BASIS_EVENT8: 8, BASIS_WMONO10: 10}


def rng_for(config_index: int, salt: int = 0) -> np.random.Generator:
    """Generator of config `config_index` (0-based); `salt` > 0 gives extra streams."""
    ss = np.random.SeedSequence(ROOT_SEED).spawn(8)[config_index]
    if salt:
        ss = ss.spawn(salt + 1)[salt]
    return np.random.default_rng(ss)


# ---------------------------------------------------------------- bf16 helpers
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if not np.all(np.isfinite(x)):
        raise ValueError("only finite values are rounded")
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------- geometry
def sphere_points(rng: np.random.Generator, n: int) -> np.ndarray:
    g = rng.standard_normal((n, 3))
    g /= np.linalg.norm(g, axis=1, keepdims=True)
    return g.astype(np.float32)


def ellipsoid_surface_points(rng: np.random.Generator, n: int, axes) -> np.ndarray:
    """Uniform-by-area samples on the surface of an axis-aligned ellipsoid.

    A direction u is drawn uniformly on the unit sphere and mapped to
    (a ux, b uy, c uz); it is kept with probability g(u)/max g, where
    g(u) = |(bc ux, ac uy, ab uz)| is the area stretch of that map.
    """
    a, b, c = (float(s) for s in axes)
    gmax = max(b * c, a * c, a * b)
    out = []
    have = 0
    while have < n:
        u = rng.standard_normal((4 * n, 3))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        g = np.sqrt((b * c * u[:, 0]) ** 2 + (a * c * u[:, 1]) ** 2 + (a * b * u[:, 2]) ** 2)
        keep = rng.random(4 * n) * gmax < g
        pts = u[keep] * np.array([a, b, c])
        out.append(pts)
        have += len(pts)
    return np.concatenate(out)[:n].astype(np.float32)


def farthest_point_indices(rng: np.random.Generator, x: np.ndarray, k: int) -> np.ndarray:
    """Iterative farthest-point selection of k indices (input selection only).

    Starts from a seeded random index, then repeatedly takes the point whose
    squared distance (float64 on the float32 coordinates) to the chosen set is
    largest, lowest index on ties.  Used only to pick the output cloud of the
    down-sampling workload.
    """
    xd = x.astype(np.float64)
    n = len(xd)
    first = int(rng.integers(n))
    chosen = [first]
    dmin = np.sum((xd - xd[first]) ** 2, axis=1)
    for _ in range(k - 1):
        nxt = int(np.argmax(dmin))          # argmax returns the lowest index on ties
        chosen.append(nxt)
        dmin = np.minimum(dmin, np.sum((xd - xd[nxt]) ** 2, axis=1))
    return np.asarray(chosen, dtype=np.int64)


# ---------------------------------------------------------------- dense tensors
def normal_f32(rng, shape, std=1.0) -> np.ndarray:
    return (rng.standard_normal(shape) * std).astype(np.float32)


def _features(rng, n_in, n_out, M, c_in, c_out, dtype):
    F = normal_f32(rng, (n_in, c_in))
    W = normal_f32(rng, (M, c_in, c_out), 1.0 / np.sqrt(M * c_in))
    dY = normal_f32(rng, (n_out, c_out))
    out = {"dtype": dtype}
    if dtype == "bf16":
        for name, arr in (("F", F), ("W", W), ("dY", dY)):
            bits = f32_to_bf16_bits(arr)
            out[name + "_bits"] = bits
            out[name] = bf16_bits_to_f32(bits)
    else:
        out.update(F=F, W=W, dY=dY)
    return out


# ---------------------------------------------------------------- workloads
def points_workload(rng, clouds, basis, radius, k_cap, c_in, c_out, dtype="f32", name=""):
    """Assemble a ragged point-cloud batch from a list of (x_in, x_out) pairs."""
    x_in = np.concatenate([c[0] for c in clouds]).astype(np.float32)
    x_out = np.concatenate([c[1] for c in clouds]).astype(np.float32)
    in_splits = np.concatenate([[0], np.cumsum([len(c[0]) for c in clouds])]).astype(np.int32)
    out_splits = np.concatenate([[0], np.cumsum([len(c[1]) for c in clouds])]).astype(np.int32)
    M = BASIS_M[basis]
    w = dict(kind="points", name=name, x_in=np.ascontiguousarray(x_in),
             x_out=np.ascontiguousarray(x_out), in_splits=in_splits, out_splits=out_splits,
             radius=float(radius), k_cap=int(k_cap), basis=basis, M=M,
             C_in=c_in, C_out=c_out, n_in=len(x_in), n_out=len(x_out))
    w.update(_features(rng, len(x_in), len(x_out), M, c_in, c_out, dtype))
    return w


def sphere_cloud(seed_index=0, n=1024, n_out=256, radius=0.2, k_cap=16, c_in=16, c_out=32,
                 basis=BASIS_MONO4):
    """One cloud uniform on the unit sphere; outputs are the first n_out inputs."""
    rng = rng_for(seed_index)
    x = sphere_points(rng, n)
    return points_workload(rng, [(x, x[:n_out])], basis, radius, k_cap, c_in, c_out,
                           name=f"sphere{n}to{n_out}")


def ellipsoid_batch(seed_index=1, n_clouds=32, n=1024, n_out=None, radius=0.1, k_cap=32,
                    c_in=64, c_out=64, basis=BASIS_MONO8, dtype="f32"):
    """n_clouds clouds uniform on ellipsoid surfaces (semi-axes U[0.5, 1]).

    n_out None: in-place (outputs = inputs); otherwise n_out outputs per cloud
    chosen by farthest-point selection.
    """
    rng = rng_for(seed_index)
    clouds = []
    for _ in range(n_clouds):
        axes = rng.uniform(0.5, 1.0, size=3)
        x = ellipsoid_surface_points(rng, n, axes)
        if n_out is None:
            clouds.append((x, x))
        else:
            idx = farthest_point_indices(rng, x, n_out)
            clouds.append((x, x[idx]))
    tag = "inplace" if n_out is None else f"down{n_out}"
    return points_workload(rng, clouds, basis, radius, k_cap, c_in, c_out, dtype,
                           name=f"ellipsoids{n_clouds}x{n}_{tag}")


def uniform_events(rng, n, width, height, duration_us):
    t = np.sort(rng.integers(0, duration_us, size=n)).astype(np.int32)
    px = rng.integers(0, width, size=n).astype(np.int32)
    py = rng.integers(0, height, size=n).astype(np.int32)
    pol = (rng.integers(0, 2, size=n) * 2 - 1).astype(np.int8)
    return px, py, t, pol


def bursty_events(rng, n, width, height, duration_us, bin_us=1000, burst=8.0,
                  p_on=1.0 / 15.0, p_off=1.0 / 5.0):
    """Events from an on/off Markov-modulated rate over fixed time bins.

    Each bin is 'on' (rate `burst`) or 'off' (rate 1); the state flips with
    probability p_on (off->on) or p_off (on->off) per bin, the first state is
    drawn from the chain's stationary law.  Bin counts are multinomial over the
    normalised rates, times are uniform integers inside a bin, then sorted.
    """
    n_bins = duration_us // bin_us
    on = np.empty(n_bins, dtype=bool)
    on[0] = rng.random() < p_on / (p_on + p_off)
    flips = rng.random(n_bins)
    for b in range(1, n_bins):
        on[b] = (flips[b] >= p_off) if on[b - 1] else (flips[b] < p_on)
    rate = np.where(on, burst, 1.0)
    counts = rng.multinomial(n, rate / rate.sum())
    t = np.concatenate([b * bin_us + rng.integers(0, bin_us, size=c) for b, c in enumerate(counts)])
    t = np.sort(t).astype(np.int32)
    px = rng.integers(0, width, size=n).astype(np.int32)
    py = rng.integers(0, height, size=n).astype(np.int32)
    pol = (rng.integers(0, 2, size=n) * 2 - 1).astype(np.int8)
    return px, py, t, pol


def event_decay_rates(n_decays, window_us):
    """Decay rates lambda_uv of the learned-decay kernel, [8, n_decays]: the
    v-th decay is 2^v / window, spread by up to 1/2 over the offsets u."""
    u = np.arange(8)[:, None]
    v = np.arange(n_decays)[None, :]
    return ((2.0 ** v) * (1.0 + u / 16.0) / float(window_us)).astype(np.float32)


def events_workload(rng, px, py, t, pol, width, height, window_us, c_in, c_out,
                    dtype="f32", name="", n_decays=1):
    """n_decays > 1: the kernel with learned decays (M_v = n_decays per offset)."""
    n = len(t)
    M = 8 * n_decays
    w = dict(kind="events", name=name, px=px, py=py, t=t, pol=pol, width=int(width),
             height=int(height), window=int(window_us), tau=float(window_us), half_extent=1,
             basis=BASIS_EVENT8 if n_decays == 1 else BASIS_EVENT_DECAYS, M=M,
             C_in=c_in, C_out=c_out, n_in=n, n_out=n)
    if n_decays > 1:
        w["decays"] = event_decay_rates(n_decays, window_us)
    w.update(_features(rng, n, n, M, c_in, c_out, dtype))
    return w


def event_stream(seed_index=3, n=300_000, width=128, height=128, duration_us=100_000,
                 window_us=10_000, c=32, dtype="f32", n_decays=1):
    rng = rng_for(seed_index)
    px, py, t, pol = uniform_events(rng, n, width, height, duration_us)
    return events_workload(rng, px, py, t, pol, width, height, window_us, c, c, dtype,
                           name=f"events{n}_{width}x{height}", n_decays=n_decays)


def bursty_event_stream(seed_index=4, n=1_000_000, width=346, height=260,
                        duration_us=200_000, window_us=5_000, c=64, dtype="bf16"):
    rng = rng_for(seed_index)
    px, py, t, pol = bursty_events(rng, n, width, height, duration_us)
    return events_workload(rng, px, py, t, pol, width, height, window_us, c, c, dtype,
                           name=f"bursty_events{n}_{width}x{height}")


# The five workloads the library is measured and checked on.
def sphere_1024():
    """1024 points on the unit sphere -> first 256; r 0.2, cap 16, M 4, 16 -> 32."""
    return sphere_cloud()


def ellipsoids_inplace():
    """32 x 1024 ellipsoid-surface points, in place; r 0.1, cap 32, M 8, 64 -> 64."""
    return ellipsoid_batch(seed_index=1)


def ellipsoids_down():
    """32 x 1024 -> 32 x 256 (farthest-point); r 0.2, cap 32, M 8, 64 -> 128."""
    return ellipsoid_batch(seed_index=2, n_out=256, radius=0.2, c_in=64, c_out=128)


def events_300k():
    """300k uniform events on 128x128 over 100 ms; 3x3, 10 ms; M 8; 32 -> 32 fp32."""
    return event_stream()


def events_1m_bf16():
    """1M bursty events on 346x260 over 200 ms; 3x3, 5 ms; M 8; 64 -> 64 bf16."""
    return bursty_event_stream()


def ellipsoids_weighted():
    """The in-place ellipsoid batch with the weighted convolution and M = 10:
    32 clouds x 1024 points, r 0.1, cap 32, 64 -> 64 fp32."""
    return ellipsoid_batch(seed_index=7, basis=BASIS_WMONO10)


def ellipsoids_featureless():
    """The paper's first layer on the in-place ellipsoid batch: a featureless
    convolution (F = 1) with the weighted M = 10 basis, 32 clouds x 1024 points,
    r 0.1, cap 32, 32 output channels.  Phi_0 is W[:, 0, :] and dZ is dY."""
    w = ellipsoid_batch(seed_index=7, basis=BASIS_WMONO10, c_in=1, c_out=32)
    w["featureless"] = True
    w["name"] = "ellipsoids32x1024_featureless"
    return w


def ellipsoids_sampling():
    """Down-sampling the ellipsoid batch for the next layer: the uncapped
    in-place ball (r 0.1) of 32 clouds x 1024 points, then rejection sampling
    and the approximate farthest points up to 256 points per cloud."""
    w = ellipsoid_batch(seed_index=1, k_cap=0)
    w["sampling"] = {"method": "approx_ifp_rejection", "per_cloud": 256}
    w["name"] = "ellipsoids32x1024_sampling"
    return w


def events_300k_decays2():
    """The 300k-event stream with learned decays, M_v = 2 per offset (M = 16)."""
    return event_stream(n_decays=2)


def events_300k_lif():
    """The next, coarser stream of the 300k-event 128x128 stream by leaky
    integrate-and-fire: 3x3 receptive fields, stride 2 (a 64x64 grid), decay
    time 4 ms, threshold 1.6, reset -3 (the CIFAR10-DVS settings of the
    supplementary's dataset table)."""
    rng = rng_for(3)
    px, py, t, _ = uniform_events(rng, 300_000, 128, 128, 100_000)
    return dict(kind="lif", name="lif300k_128x128", px=px, py=py, t=t, width=128, height=128,
                kernel=3, stride=2, decay=4000.0, v_thresh=1.6, v_reset=-3.0, n_in=len(t),
                dtype="f64")


def events_stream():
    """The 300k-event 128x128 stream through the convolution's deployment form
    (per-pixel decayed sums, Eq. 13-15) in batches of 4096 events: tau 10 ms,
    32 -> 32 channels fp32, the state carried from batch to batch."""
    w = event_stream()
    w["batch"] = 4096
    w["kind"] = "stream"
    w["name"] = "stream300k_128x128"
    return w


def table2_flexconv():
    """The operator benchmark shape of the paper's Table 2: 8 clouds x 4096
    points (uniform in the unit cube; the table gives no distribution), in
    place, the 9 nearest (the point itself included) within r = 0.25, which
    always holds at least 9 (E = 294,912); M 4; 64 -> 64 channels fp32.  Like
    the table, the step leaves out the neighbour search."""
    rng = rng_for(7, salt=1)
    clouds = []
    for _ in range(8):
        x = rng.uniform(0.0, 1.0, size=(4096, 3))
        clouds.append((x, x))
    w = points_workload(rng, clouds, BASIS_MONO4, 0.25, 9, 64, 64, name="table2_8x4096")
    w["search_in_step"] = False
    return w


WORKLOADS = {
    "sphere_1024": sphere_1024,
    "ellipsoids_inplace": ellipsoids_inplace,
    "ellipsoids_down": ellipsoids_down,
    "events_300k": events_300k,
    "events_1m_bf16": events_1m_bf16,
    "ellipsoids_weighted": ellipsoids_weighted,
    "ellipsoids_featureless": ellipsoids_featureless,
    "events_300k_decays2": events_300k_decays2,
    "ellipsoids_sampling": ellipsoids_sampling,
    "events_300k_lif": events_300k_lif,
    "events_stream": events_stream,
    "table2_flexconv": table2_flexconv,
}


def small_events(seed=0, n=4000, width=20, height=16, duration_us=20_000, window_us=3000,
                 c=8, dtype="f32", n_decays=1):
    """A small uniform stream for tests (several tiles, ragged tail)."""
    rng = rng_for(5, salt=seed + 1)
    px, py, t, pol = uniform_events(rng, n, width, height, duration_us)
    return events_workload(rng, px, py, t, pol, width, height, window_us, c, c, dtype,
                           name=f"small_events{n}", n_decays=n_decays)


def small_points(seed=0, n_clouds=3, n=300, n_out=None, radius=0.25, k_cap=12, c_in=8,
                 c_out=12, basis=BASIS_MONO8, dtype="f32"):
    """A small ragged batch for tests: clouds of different sizes on ellipsoids."""
    rng = rng_for(6, salt=seed + 1)
    clouds = []
    for b in range(n_clouds):
        nb = n + 37 * b
        axes = rng.uniform(0.5, 1.0, size=3)
        x = ellipsoid_surface_points(rng, nb, axes)
        if n_out is None:
            clouds.append((x, x))
        else:
            idx = farthest_point_indices(rng, x, n_out + 5 * b)
            clouds.append((x, x[idx]))
    return points_workload(rng, clouds, basis, radius, k_cap, c_in, c_out, dtype,
                           name=f"small_points{n_clouds}x{n}")
