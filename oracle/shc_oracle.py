"""CPU oracle for the sparse contact-layer operators -- TEST INFRASTRUCTURE ONLY.

Only the tests, the package's smoke check and the benchmark's CPU-baseline leg
may import this module.  The library's product path never calls it, and it
shares no code with the HIP kernels (no common helpers, tables or constants).

What it computes (Sec. 3.1-3.2 of the paper, arXiv 2608.09388):

* Eq. 1: the contact mask multiplies the per-vertex input elementwise.  The
  mask is per vertex and broadcast over channels; masks are given per body /
  frame b, so ``m`` is [B][V].
* Eq. 2: the masked tensor is decomposed into a coordinate list C' of
  (frame b, vertex x) pairs and the feature rows S' of the non-zero entries.
  The list order is (b, x) ascending (the paper leaves it open).
* Eqs. 4-5: a sparse convolution produces output only at the active centre
  coordinate and sums, over the kernel slots, the slot weight times the
  feature of the neighbour that slot points at, where that neighbour is
  present in C_k.  On a mesh the slots are the 9 neighbour positions of
  ``nbr[v]``; every slot carries a C_in x C_out channel-mixing matrix W[j]
  (the paper's scalar slot weight is the special case W[j] = w_j * I).
* Eq. 6: the sparse linear layer maps each feature row through W_l and adds
  b; coordinates are unchanged.
* Eq. 10: an activation acts elementwise on the feature rows.
* Pooling is named alongside the other sparse layers but not defined; here
  it is the maximum over the active rows of each body / frame, 0 for a body
  with no active row.
* Sec. 3.1 (several masks): each mask k of a set of kappa is applied to the
  same input independently.  Stacked as a batch axis, body b under mask k is
  body b' = k * B + b of a [kappa * B][V] mask whose rows read the input of
  body b' mod B; the kappa outputs are then combined by a rule the paper
  leaves open (sum, mean or maximum here).  A mask drawn per element
  (vertex and channel) makes a vertex active when any of its channels is
  kept, and multiplies the gathered row by the element mask.
* Eq. 3: the mask score.  For K masks with aligned outputs O_k (one row per
  vertex and body, C channels), the similarity of masks i and k is
  ||O_i^T O_k||_F^2 / (||O_k^T O_k||_F ||O_i^T O_i||_F), and alpha_k grows by
  the mean over i != k of (1 - similarity).  At inference the kappa masks of
  largest alpha are kept (ties to the lower index).
* Backward of the sparse linear and conv layers: the gradient of the dense
  operator on x (.) m, restricted to the active rows (input rows, slot
  weights, bias), with the activation's derivative taken from the stored
  output.
* Eqs. 7-9: sparse group normalization.  The channels are split into G
  groups of C/G; for every body / frame b and group g the mean and the
  (biased, 1/N) variance are taken over the group's values in the ACTIVE rows
  of b only, and those values are centred and divided by sqrt(var + eps).
  No affine term; eps = 1e-5 unless given.  G = 1 is layer normalization.

Every layer but the normalization is computed the plain way: the DENSE
operator is applied to the masked input x (.) m on all B*V rows in fp64, and
the result is then read at the active rows.  Since a sparse operator only ever
reads active rows, this restriction is exactly the sparse operator's result
(up to rounding order).  Group normalization is the exception: the dense
operator on x (.) m would let the inactive rows' zeros into the statistics,
so it is written out per body and group over the active rows, as Eqs. 7-9
define it.

Precision: inputs are widened exactly to fp64 and all sums are fp64.  For
bfloat16 stacks each layer output is rounded to bfloat16 (round to nearest,
ties to even) by :func:`round_bf16` before it feeds the next layer, which is
how bfloat16 activations are stored between layers.
"""
from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------
# Eq. 2: decomposition of the masked tensor into (C', S')
# ----------------------------------------------------------------------------


def compact(mask: np.ndarray):
    """Decompose a [B][V] 0/1 mask (Eq. 2).

    Returns ``coords`` int32 [N'][2] of (b, v) in row-major order, ``inv``
    int32 [B*V] (row index of (b, v) in C', or -1 when inactive), ``row_ptr``
    int32 [B+1] (first row of body b; row_ptr[B] = N'), and N'.

    An entry is active when it is non-zero.  Row i of C' is the i-th active
    entry in row-major order, so its index is the number of active entries
    before it: an exclusive running count.
    """
    m = np.asarray(mask)
    B, V = m.shape
    active = (m.reshape(-1) != 0)
    count_before = np.cumsum(active, dtype=np.int64) - active   # exclusive count
    n = int(active.sum())
    inv = np.where(active, count_before, -1).astype(np.int32)
    flat = np.arange(B * V, dtype=np.int64)
    coords = np.empty((n, 2), dtype=np.int32)
    coords[count_before[active], 0] = flat[active] // V
    coords[count_before[active], 1] = flat[active] % V
    # body b starts after every active entry that precedes its first element
    row_ptr = np.empty(B + 1, dtype=np.int32)
    row_ptr[:B] = count_before[np.arange(B, dtype=np.int64) * V]
    row_ptr[B] = n
    return coords, inv, row_ptr, n


def gather(x: np.ndarray, coords: np.ndarray, V: int) -> np.ndarray:
    """S'[i] = x[b_i, v_i]: the feature rows of the active coordinates (Eq. 2)."""
    x = np.asarray(x)
    flat = coords[:, 0].astype(np.int64) * V + coords[:, 1].astype(np.int64)
    return x[flat]


def densify(S: np.ndarray, coords: np.ndarray, B: int, V: int) -> np.ndarray:
    """The masked dense tensor x (.) m rebuilt from (C', S'): zeros at inactive rows."""
    S = np.asarray(S)
    D = np.zeros((B * V, S.shape[1]), dtype=S.dtype)
    flat = coords[:, 0].astype(np.int64) * V + coords[:, 1].astype(np.int64)
    D[flat] = S
    return D


# ----------------------------------------------------------------------------
# dense operators (fp64) applied to the masked input
# ----------------------------------------------------------------------------


def dense_linear(xm: np.ndarray, W: np.ndarray, bias=None) -> np.ndarray:
    """Eq. 6 on every row: y = x W + b  (W is [C_in][C_out]), fp64."""
    y = np.asarray(xm, dtype=np.float64) @ np.asarray(W, dtype=np.float64)
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)[None, :]
    return y


def dense_conv(xm: np.ndarray, nbr: np.ndarray, W: np.ndarray, B: int, V: int,
               bias=None) -> np.ndarray:
    """Eqs. 4-5 on every vertex of every body, fp64.

    y[b, v] = bias + sum over slots j with nbr[v, j] >= 0 of x[b, nbr[v, j]] W[j],
    with W [K][C_in][C_out].  A slot whose neighbour index is -1 adds nothing.
    ``xm`` is the masked input (inactive rows zero), so an inactive neighbour
    also adds nothing -- only neighbours present in C_k contribute.
    """
    x = np.asarray(xm, dtype=np.float64).reshape(B, V, -1)
    W = np.asarray(W, dtype=np.float64)
    K = W.shape[0]
    y = np.zeros((B, V, W.shape[2]), dtype=np.float64)
    for j in range(K):
        n_j = nbr[:, j].astype(np.int64)
        has = n_j >= 0
        contrib = x[:, np.where(has, n_j, 0), :] @ W[j]       # [B][V][C_out]
        y += np.where(has[None, :, None], contrib, 0.0)
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)[None, None, :]
    return y.reshape(B * V, -1)


def relu(y: np.ndarray) -> np.ndarray:
    """Eq. 10 with f_act = ReLU: y if y > 0 else 0 (NaN maps to 0)."""
    return np.where(y > 0, y, 0.0)


def restrict(yd: np.ndarray, coords: np.ndarray, V: int) -> np.ndarray:
    """Read a dense result at the active coordinates (C' unchanged, Eqs. 5-6, 10)."""
    return gather(yd, coords, V)


# ----------------------------------------------------------------------------
# sparse layers by their definition: dense op on x (.) m, then restriction
# ----------------------------------------------------------------------------


def sparse_linear(S, coords, B, V, W, bias=None, act=False):
    """Sparse linear layer on the active rows S (Eq. 6 [+ Eq. 10])."""
    y = dense_linear(densify(np.asarray(S, np.float64), coords, B, V), W, bias)
    if act:
        y = relu(y)
    return restrict(y, coords, V)


def sparse_conv(S, coords, B, V, nbr, W, bias=None, act=False):
    """Sparse neighbourhood convolution on the active rows S (Eqs. 4-5 [+ Eq. 10])."""
    y = dense_conv(densify(np.asarray(S, np.float64), coords, B, V), nbr, W, B, V, bias)
    if act:
        y = relu(y)
    return restrict(y, coords, V)


def sparse_conv_scale(S, coords, B, V, nbr, W, bias=None):
    """Abs-sum of every output's dot product over all slots (error scale)."""
    return sparse_conv(np.abs(np.asarray(S, np.float64)), coords, B, V, nbr, np.abs(W),
                       None if bias is None else np.abs(bias))


def conv_at(S, coords, B, V, nbr, W, rows, bias=None, act=False, scale=False):
    """Eqs. 4-5 evaluated at selected active rows only (for full-size checks).

    Same definition as :func:`sparse_conv`: the dense convolution of the
    masked input, read at the centre coordinates (b_i, v_i) of the selected
    rows ``rows``.  The masked input at (b, u) is the C' feature row of
    (b, u) when that coordinate is in C', else zero.  With ``scale`` the
    abs-sum error scale is returned instead of the output.
    """
    S = np.asarray(S)
    rows = np.asarray(rows, dtype=np.int64)
    n = S.shape[0]
    W = np.asarray(W, dtype=np.float64)
    if scale:
        W = np.abs(W)
    K, _, Cout = W.shape
    where = np.full(B * V, -1, dtype=np.int64)         # coordinate -> row of C'
    where[coords[:, 0].astype(np.int64) * V + coords[:, 1]] = np.arange(n)
    b = coords[rows, 0].astype(np.int64)
    v = coords[rows, 1].astype(np.int64)
    y = np.zeros((rows.size, Cout), dtype=np.float64)
    for j in range(K):
        u = nbr[v, j].astype(np.int64)
        r = np.where(u >= 0, where[b * V + np.maximum(u, 0)], -1)
        xm = np.where((r >= 0)[:, None], S[np.maximum(r, 0)].astype(np.float64), 0.0)
        if scale:
            xm = np.abs(xm)
        y += xm @ W[j]
    if bias is not None:
        y += np.abs(bias) if scale else np.asarray(bias, dtype=np.float64)
    if act and not scale:
        y = relu(y)
    return y


def linear_at(S, W, rows, bias=None, act=False, scale=False):
    """Eq. 6 at selected rows (row i of the result depends on S[i] only)."""
    rows = np.asarray(rows, dtype=np.int64)
    x = np.asarray(S)[rows].astype(np.float64)
    W = np.asarray(W, dtype=np.float64)
    if scale:
        x, W = np.abs(x), np.abs(W)
    y = x @ W
    if bias is not None:
        y += np.abs(bias) if scale else np.asarray(bias, dtype=np.float64)
    if act and not scale:
        y = relu(y)
    return y


def scatter(S: np.ndarray, inv: np.ndarray, zero_fill: bool = True, D=None) -> np.ndarray:
    """Compact rows back to the dense [B*V] layout: D[r] = S[inv[r]] if active.

    With zero_fill, inactive rows become 0 (this is y (.) m); otherwise they
    keep the contents of ``D``.
    """
    S = np.asarray(S)
    if D is None:
        D = np.zeros((inv.shape[0], S.shape[1]), dtype=S.dtype)
    else:
        D = np.array(D, copy=True)
    act = inv >= 0
    if zero_fill:
        D[~act] = 0
    D[act] = S[inv[act]]
    return D


def segment_max(S: np.ndarray, row_ptr: np.ndarray, empty_value: float = 0.0) -> np.ndarray:
    """Per-body maximum over its active rows (the paper's sparse pooling).

    P[b, c] = max over row_ptr[b] <= i < row_ptr[b+1] of S[i, c], ignoring NaN
    (IEEE maxNum), and ``empty_value`` for a body with no active row.
    """
    S = np.asarray(S)
    B = row_ptr.shape[0] - 1
    P = np.full((B, S.shape[1]), empty_value, dtype=S.dtype)
    for b in range(B):
        lo, hi = int(row_ptr[b]), int(row_ptr[b + 1])
        if hi > lo:
            P[b] = np.fmax.reduce(S[lo:hi], axis=0)
    return P


# ----------------------------------------------------------------------------
# Sec. 3.1: several masks (stacked as a batch axis), per-element masks
# ----------------------------------------------------------------------------


def stack_masks(masks: np.ndarray) -> np.ndarray:
    """[kappa][B][V] masks -> one [kappa * B][V] mask: row k * B + b is mask k
    of body b."""
    m = np.asarray(masks)
    k, B, V = m.shape
    return m.reshape(k * B, V)


def gather_stacked(x: np.ndarray, coords: np.ndarray, B: int, V: int) -> np.ndarray:
    """Rows of the stacked batch: row (b', v) reads the input of body b' mod B."""
    b = coords[:, 0].astype(np.int64) % B
    return np.asarray(x)[b * V + coords[:, 1].astype(np.int64)]


def combine_stacked(Y: np.ndarray, kappa: int, op: str) -> np.ndarray:
    """Combine kappa stacked outputs [kappa * R][C] -> [R][C], row by row and
    channel by channel: 'sum', 'mean' or 'max' over k of Y[k * R + r]."""
    Y = np.asarray(Y, dtype=np.float64)
    R = Y.shape[0] // kappa
    out = Y[:R].copy()
    for k in range(1, kappa):
        blk = Y[k * R:(k + 1) * R]
        out = np.maximum(out, blk) if op == "max" else out + blk
    if op == "mean":
        out = out / kappa
    elif op not in ("sum", "max"):
        raise ValueError(op)
    return out


def row_mask_from_elements(me: np.ndarray) -> np.ndarray:
    """Per-element mask [B][V][C] -> per-vertex activity [B][V]: a vertex is
    active when any of its channels is kept."""
    return (np.asarray(me) != 0).any(axis=2).astype(np.uint8)


def gather_masked(x: np.ndarray, me: np.ndarray, coords: np.ndarray, V: int) -> np.ndarray:
    """Active rows of the element-masked input: x[b, v, c] where the element
    mask keeps (b, v, c), else 0."""
    rows = coords[:, 0].astype(np.int64) * V + coords[:, 1].astype(np.int64)
    C = np.asarray(x).shape[-1]
    keep = (np.asarray(me).reshape(-1, C)[rows] != 0)
    return np.where(keep, np.asarray(x)[rows], 0)


# ----------------------------------------------------------------------------
# Eq. 3: mask scores and top-kappa selection
# ----------------------------------------------------------------------------


def gram_frobenius(O: np.ndarray) -> np.ndarray:
    """F[i][k] = ||O_i^T O_k||_F^2 for outputs O [K][N][C] (fp64)."""
    O = np.asarray(O, dtype=np.float64)
    K = O.shape[0]
    F = np.empty((K, K))
    for i in range(K):
        for k in range(K):
            G = O[i].T @ O[k]
            F[i, k] = float((G * G).sum())
    return F


def mask_similarity(O: np.ndarray) -> np.ndarray:
    """sim[i][k] = ||O_i^T O_k||_F^2 / (||O_k^T O_k||_F ||O_i^T O_i||_F) (Eq. 3).

    Eq. 3 leaves the quotient undefined when one of the two outputs is all
    zero.  Such a mask adds nothing beyond the others, so it is given no
    dissimilarity credit: the similarity of a pair with a zero output is 1
    (which is also every output's similarity with itself)."""
    F = gram_frobenius(O)
    d = np.sqrt(np.diag(F))
    den = np.outer(d, d)
    return np.where(den > 0, F / np.where(den > 0, den, 1.0), 1.0)


def alpha_update(alpha: np.ndarray, O: np.ndarray) -> np.ndarray:
    """One step of Eq. 3: alpha_k + 1/(K-1) sum_{i != k} (1 - sim[i][k]).

    The paper always has several masks; with K = 1 the sum is empty and the
    score is left as it is (the 1/(K-1) factor is not applied)."""
    sim = mask_similarity(O)
    K = sim.shape[0]
    out = np.array(alpha, dtype=np.float64, copy=True)
    if K == 1:
        return out
    for k in range(K):
        out[k] += sum(1.0 - sim[i, k] for i in range(K) if i != k) / (K - 1)
    return out


def top_kappa(alpha: np.ndarray, kappa: int) -> np.ndarray:
    """Indices of the kappa largest scores, largest first; ties to the lower index."""
    a = np.asarray(alpha, dtype=np.float64)
    order = sorted(range(len(a)), key=lambda k: (-a[k], k))
    return np.array(order[:kappa], dtype=np.int32)


# ----------------------------------------------------------------------------
# backward of the sparse linear and conv layers
# ----------------------------------------------------------------------------
#
# A sparse layer is the dense layer applied to x (.) m and read at the active
# rows: out = R L(P^T S), where P^T places the active rows S into a zero
# dense tensor, L is the dense operator and R reads the active rows.  With the
# upstream gradient dY at the output rows, the chain rule gives
#   dZ = dY (.) f'(Z)                      (Eq. 10; for ReLU, [Y > 0])
#   dS = P L^T(R^T dZ)                     (input rows)
#   dW, db: the dense layer's weight gradients at R^T dZ,
# i.e. the gradient of the dense operator on x (.) m, restricted to the
# active rows.  The ReLU's derivative is taken from the layer's stored output
# Y (derivative 0 at 0), so it is an input here, not recomputed.


def relu_backward(dY: np.ndarray, Y: np.ndarray) -> np.ndarray:
    """Gradient through Eq. 10's ReLU from the stored output: dY where Y > 0, else 0."""
    dY = np.asarray(dY, dtype=np.float64)
    return np.where(np.asarray(Y, dtype=np.float64) > 0, dY, 0.0)


def dense_conv_transpose(dZd: np.ndarray, nbr: np.ndarray, W: np.ndarray, B: int,
                         V: int) -> np.ndarray:
    """Adjoint of :func:`dense_conv` in x: each output row (b, v) sends
    dZ[b, v] W[j]^T back to its slot-j neighbour (b, nbr[v, j]), fp64."""
    dZ = np.asarray(dZd, dtype=np.float64).reshape(B, V, -1)
    W = np.asarray(W, dtype=np.float64)
    K, Cin = W.shape[0], W.shape[1]
    dX = np.zeros((B, V, Cin), dtype=np.float64)
    for j in range(K):
        n_j = nbr[:, j].astype(np.int64)
        has = np.flatnonzero(n_j >= 0)
        contrib = dZ[:, has, :] @ W[j].T                     # [B][|has|][C_in]
        for b in range(B):
            np.add.at(dX[b], n_j[has], contrib[b])
    return dX.reshape(B * V, Cin)


def sparse_linear_backward(S, W, dY, Y=None, act=False):
    """Gradients of the sparse linear layer (Eq. 6 [+ Eq. 10]).

    Rows are independent, so the dense gradient read at the active rows is
    dZ = dY (.) [Y > 0] (with the activation), dS = dZ W^T, dW = S^T dZ,
    db = sum of dZ over the rows.  Returns (dS, dW, db) in fp64."""
    S = np.asarray(S, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    dZ = relu_backward(dY, Y) if act else np.asarray(dY, dtype=np.float64)
    return dZ @ W.T, S.T @ dZ, dZ.sum(axis=0)


def sparse_conv_backward(S, coords, B, V, nbr, W, dY, Y=None, act=False):
    """Gradients of the sparse neighbourhood convolution (Eqs. 4-5 [+ Eq. 10]).

    The output gradient is placed in a zero dense tensor (inactive output rows
    receive none), sent back through the adjoint of the dense convolution and
    read at the active rows; the slot weights' gradient is the dense one,
    dW[j] = sum over dense rows (b, v) of x_m[b, nbr[v, j]]^T dZ[b, v], where
    only active rows carry a non-zero x_m and dZ.  Returns (dS, dW, db)."""
    S = np.asarray(S, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    dZ = relu_backward(dY, Y) if act else np.asarray(dY, dtype=np.float64)
    dZd = densify(dZ, coords, B, V)
    dS = restrict(dense_conv_transpose(dZd, nbr, W, B, V), coords, V)
    xm = densify(S, coords, B, V).reshape(B, V, -1)
    dZ3 = dZd.reshape(B, V, -1)
    K = W.shape[0]
    dW = np.zeros_like(W)
    for j in range(K):
        n_j = nbr[:, j].astype(np.int64)
        has = n_j >= 0
        xs = np.where(has[None, :, None], xm[:, np.where(has, n_j, 0), :], 0.0)
        dW[j] = xs.reshape(B * V, -1).T @ dZ3.reshape(B * V, -1)
    return dS, dW, dZ.sum(axis=0)


def conv_backward_weight_bias(S, coords, B, V, nbr, dZ, K, scale=False):
    """dW and db of the sparse convolution from the pre-activation gradient dZ
    of all active rows (for full-size checks, without the dense tensors).

    Slot j's weight gradient sums, over the active rows i = (b, v) whose slot-j
    neighbour u = nbr[v, j] is an active row r of the same body, the outer
    product S[r]^T dZ[i]; rows with an absent neighbour add nothing.  db sums
    dZ over the active rows.  With ``scale`` the abs-sum error scales
    (sums of |S[r]|^T |dZ[i]| and of |dZ[i]|) are returned instead."""
    S = np.asarray(S, dtype=np.float64)
    dZ = np.asarray(dZ, dtype=np.float64)
    if scale:
        S, dZ = np.abs(S), np.abs(dZ)
    n = dZ.shape[0]
    where = np.full(B * V, -1, dtype=np.int64)         # coordinate -> row of C'
    where[coords[:, 0].astype(np.int64) * V + coords[:, 1]] = np.arange(n)
    b = coords[:, 0].astype(np.int64)
    v = coords[:, 1].astype(np.int64)
    dW = np.zeros((K, S.shape[1], dZ.shape[1]), dtype=np.float64)
    for j in range(K):
        u = nbr[v, j].astype(np.int64)
        r = np.where(u >= 0, where[b * V + np.maximum(u, 0)], -1)
        has = r >= 0
        dW[j] = S[r[has]].T @ dZ[has]
    return dW, dZ.sum(axis=0)


def conv_backward_input_at(coords, B, V, nbr, W, dZ, rows, scale=False):
    """dS of the sparse convolution at selected active rows only, from the
    pre-activation gradient dZ of all active rows (for full-size checks).

    Row r = (b, u) receives dZ[b, v] W[j]^T from every active (b, v) whose
    slot j points at u.  With ``scale`` the abs-sum error scale is returned."""
    rows = np.asarray(rows, dtype=np.int64)
    dZ = np.asarray(dZ, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    if scale:
        W, dZ = np.abs(W), np.abs(dZ)
    n = dZ.shape[0]
    where = np.full(B * V, -1, dtype=np.int64)
    where[coords[:, 0].astype(np.int64) * V + coords[:, 1]] = np.arange(n)
    out = np.zeros((rows.size, W.shape[1]), dtype=np.float64)
    for q, r in enumerate(rows):
        b, u = int(coords[r, 0]), int(coords[r, 1])
        for j in range(W.shape[0]):
            for v in np.flatnonzero(nbr[:, j] == u):
                i = where[b * V + v]
                if i >= 0:
                    out[q] += dZ[i] @ W[j].T
    return out


# ----------------------------------------------------------------------------
# Eqs. 7-9: sparse group normalization
# ----------------------------------------------------------------------------


def group_norm(S: np.ndarray, row_ptr: np.ndarray, G: int, eps: float = 1e-5) -> np.ndarray:
    """Sparse group normalization of the active rows (Eqs. 7-9).

    ``S`` [N'][C] holds the active rows of every body in order, ``row_ptr``
    [B+1] the first row of each body.  For body b and channel group g (C/G
    consecutive channels), mu is the mean and var the mean squared deviation
    of the group's values over the rows of b (Eqs. 7 and 8); each value
    becomes (value - mu) / sqrt(var + eps) (Eq. 9).  A body without rows has
    nothing to normalize.  Computed in fp64.
    """
    S = np.asarray(S, dtype=np.float64)
    n, C = S.shape
    if C % G != 0:
        raise ValueError(f"C = {C} is not a multiple of G = {G}")
    cg = C // G
    out = np.empty_like(S)
    for b in range(len(row_ptr) - 1):
        lo, hi = int(row_ptr[b]), int(row_ptr[b + 1])
        if hi <= lo:
            continue
        for g in range(G):
            vals = S[lo:hi, g * cg:(g + 1) * cg]
            mu = vals.mean()
            var = ((vals - mu) ** 2).mean()
            out[lo:hi, g * cg:(g + 1) * cg] = (vals - mu) / np.sqrt(var + eps)
    return out


# ----------------------------------------------------------------------------
# bfloat16 rounding (storage of bf16 activations between layers)
# ----------------------------------------------------------------------------

_BF16_SIG_BITS = 8            # 1 implicit + 7 stored significand bits
_BF16_EMIN = -126             # smallest normal exponent (shared with fp32)
_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16 value, ties to even (fp64 out).

    A bfloat16 number has 8 significant bits and fp32's exponent range.  For
    a finite x with 2^e <= |x| < 2^(e+1) the spacing of representable values
    is 2^(e-7), or 2^(-133) below the normal range; x is divided by that
    spacing, rounded half-to-even to an integer (np.rint) and scaled back.
    Results past the largest finite value round to +-inf the IEEE way: a
    value at or above max + half a spacing overflows.  NaN stays NaN.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, copy=True)
    fin = np.isfinite(x) & (x != 0)
    ax = np.abs(x[fin])
    _, e = np.frexp(ax)                      # ax = f * 2^e, 0.5 <= f < 1
    e = e - 1                                # 2^e <= ax < 2^(e+1)
    e = np.maximum(e, _BF16_EMIN)            # subnormals share the min spacing
    spacing_exp = e - (_BF16_SIG_BITS - 1)
    q = np.rint(np.ldexp(ax, -spacing_exp))  # exact scaling, RNE to integer
    r = np.ldexp(q, spacing_exp)
    overflow_at = _BF16_MAX + 2.0 ** (127 - _BF16_SIG_BITS)   # max + half spacing
    r = np.where(ax >= overflow_at, np.inf, r)
    out[fin] = np.sign(x[fin]) * r
    return out


def round_f32(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to fp32 storage (IEEE conversion, to nearest with ties
    to even; past the largest finite value to +-inf), returned as fp64."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the storage dtype ('f32' or 'bf16'); values returned as fp64."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# stacks: x^{l+1} = act(op_l(x^l (.) m)) (.) m, active set fixed (C'_k = C_k)
# ----------------------------------------------------------------------------


def run_stack(x, mask, nbr, layers, dtype: str, pool: bool = False):
    """Evaluate a whole sparse stack from the dense input and the mask.

    ``layers`` is a sequence of (kind, W, bias, relu) with kind 'conv' or
    'linear'.  Returns a dict with coords/inv/row_ptr/n, the active rows
    after every layer (stored-dtype values, fp64) and, if ``pool``, the
    per-body maximum of the last layer.
    """
    mask = np.asarray(mask)
    B, V = mask.shape
    coords, inv, row_ptr, n = compact(mask)
    S = gather(np.asarray(x, np.float64), coords, V)
    outs = []
    for kind, W, bias, act in layers:
        if kind == "conv":
            y = sparse_conv(S, coords, B, V, nbr, W, bias, act)
        elif kind == "linear":
            y = sparse_linear(S, coords, B, V, W, bias, act)
        else:
            raise ValueError(kind)
        S = store(y, dtype)
        outs.append(S)
    res = dict(coords=coords, inv=inv, row_ptr=row_ptr, n=n, outs=outs)
    if pool:
        res["pool"] = segment_max(S, row_ptr, 0.0)
    return res
