"""Float64 CPU oracle of the optimiser step: gradient clipping by the global norm, Muon on the
hidden weight matrices (its Newton-Schulz orthogonalisation batched over the Q, K and V
matrices), and schedule-free AdamW on every other parameter.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test-suite, the smoke check
and the CPU-baseline leg of the benchmark may import it, and it imports nothing from the GPU
package.

What the paper fixes (Sec. 5 "Muon Optimizer", "Batched Muon, Compile"; App. "Muon Optimizer",
"Batched Muon, Compile"; Tab. 5): Muon updates the two-dimensional hidden weight matrices of the
blocks and schedule-free AdamW everything else; the Muon learning rate is 0.1 x the AdamW one,
its momentum 0.96 and its weight decay 0.1 in the current best record; AdamW weight decay 0 in
the baseline and 0.01 in the record; gradients are clipped to a global norm of 1.0 (baseline)
or 2.0 (record); the Newton-Schulz iteration runs batched over the Q, K and V matrices.

The algorithms themselves are the published ones, written here from their definitions:

* Muon (Jordan et al. 2024, the optimiser the paper cites): heavy-ball momentum of the gradient
  with a Nesterov look-ahead, the result orthogonalised by five steps of the quintic
  Newton-Schulz map X <- a X + b (X X^T) X + c (X X^T)^2 X with (a, b, c) = (3.4445, -4.7750,
  2.0315) after scaling X to unit Frobenius norm (the map is applied to the wide orientation of
  the matrix), the weight first shrunk by (1 - lr wd), then moved by -lr max(1, rows/cols)^(1/2)
  times the orthogonalised matrix.
* Schedule-free AdamW (Defazio et al. 2024, "The Road Less Scheduled", the AdamW form of its
  Algorithm 1), three sequences: gradients are taken at y_t = (1 - b1) z_t + b1 x_t;
  v_t = b2 v_{t-1} + (1 - b2) g_t^2; with the scheduled rate s_t = lr min(1, t / warmup) and the
  step rate gamma_t = s_t sqrt(1 - b2^t),
  z_{t+1} = z_t - gamma_t (g_t / (sqrt(v_t) + eps) + wd y_t);
  x_{t+1} = (1 - c_{t+1}) x_t + c_{t+1} z_{t+1} with c_{t+1} = gamma_t^2 / sum_{i<=t} gamma_i^2
  (the averaging weights are the squared step rates, bias correction included).
  Starting point x_1 = z_1 = y_1 = the initial parameters, v_0 = 0.

Readings where the paper is silent are listed in the design doc: the Nesterov form and the momentum
average (buf <- m buf + (1 - m) g, input (1 - m) g + m buf), the Frobenius-norm guard 1e-7, the
b1 = 0.9, b2 = 0.999, eps = 1e-8, no warm-up unless given, and the clip factor
min(1, max_norm / (norm + 1e-6)).
"""

import numpy as np

NS_COEFFS = (3.4445, -4.7750, 2.0315)
NS_STEPS = 5
NS_EPS = 1e-7
CLIP_EPS = 1e-6


def clip_scale(grads, max_norm):
    """Global L2 norm of all gradient arrays and the factor that clips it to max_norm."""
    total = float(np.sqrt(sum(float(np.sum(np.asarray(g, dtype=np.float64) ** 2))
                              for g in grads)))
    return total, min(1.0, max_norm / (total + CLIP_EPS))


def newton_schulz(G, steps=NS_STEPS, coeffs=NS_COEFFS, eps=NS_EPS):
    """Quintic Newton-Schulz orthogonalisation of one matrix (float64)."""
    a, b, c = coeffs
    X = np.asarray(G, dtype=np.float64)
    tall = X.shape[0] > X.shape[1]
    if tall:
        X = X.T
    X = X / (np.linalg.norm(X) + eps)
    for _ in range(steps):
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X.T if tall else X


def muon_step(W, G, buf, lr, momentum, weight_decay, nesterov=True, steps=NS_STEPS):
    """One Muon step on a batch of equally shaped matrices W[i] with gradients G[i] and momentum
    buffers buf[i] (float64 arrays [count, rows, cols]).  Returns (W_new, buf_new)."""
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    buf = momentum * np.asarray(buf, dtype=np.float64) + (1.0 - momentum) * G
    U = (1.0 - momentum) * G + momentum * buf if nesterov else buf
    rows, cols = W.shape[-2:]
    scale = max(1.0, rows / cols) ** 0.5
    O = np.stack([newton_schulz(U[i], steps) for i in range(U.shape[0])])
    return W * (1.0 - lr * weight_decay) - lr * scale * O, buf


class ScheduleFreeAdamW:
    """The three-sequence form of schedule-free AdamW on one float64 parameter vector.  `y` is
    where the next gradient must be taken; `step(g)` consumes that gradient."""

    def __init__(self, y0, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, warmup=0):
        y0 = np.asarray(y0, dtype=np.float64)
        self.x = y0.copy()
        self.z = y0.copy()
        self.v = np.zeros_like(y0)
        self.t = 0
        self.gsq = 0.0
        self.lr, self.b1, self.b2, self.eps = lr, beta1, beta2, eps
        self.wd, self.warmup = weight_decay, warmup
        self.z_hist = [self.z.copy()]
        self.gamma_hist = []

    @property
    def y(self):
        return (1.0 - self.b1) * self.z + self.b1 * self.x

    def step(self, g):
        g = np.asarray(g, dtype=np.float64)
        y = self.y
        self.t += 1
        t = self.t
        sched = self.lr * (min(1.0, t / self.warmup) if self.warmup else 1.0)
        self.v = self.b2 * self.v + (1.0 - self.b2) * g * g
        gamma = sched * np.sqrt(1.0 - self.b2 ** t)
        self.z = self.z - gamma * (g / (np.sqrt(self.v) + self.eps) + self.wd * y)
        self.gsq += gamma * gamma
        c = gamma * gamma / self.gsq
        self.x = (1.0 - c) * self.x + c * self.z
        self.z_hist.append(self.z.copy())
        self.gamma_hist.append(gamma)
        return self.y
