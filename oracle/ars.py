"""Oracle: Adaptive Rollout Sampling controller (test infrastructure only; see
oracle/__init__).

Paper, Sec. 3.3 and Alg. 1 Phase 1(a)/(b):
* per step, the mean and the max over questions of the retained count |S(q)| are
  appended to two epoch buffers;
* at an epoch boundary: alpha = step / M (M = total steps),
  G'_t = alpha * mean(B_mean) + (1 - alpha) * mean(B_max); after the first epoch
  the reference G'_ref = (mean(B_mean) + mean(B_max)) / 2 is set once; the buffers
  are reset;
* before each step: if both G'_t and G'_ref are set and G'_t < G'_ref,
  n = max(round(min(G - (G'_ref - G'_t), G)), 2), else n = G.

Readings: Alg. 1's form is followed (the epoch statistic is the mean of per-step
maxima, not one max over the epoch); ``round`` is round-half-to-even; "step" in
alpha is the 1-based index of the step that closes the epoch.
"""


class ARSController:
    def __init__(self, G1, total_steps, steps_per_epoch):
        if G1 < 2 or total_steps < 1 or steps_per_epoch < 1:
            raise ValueError("G1 >= 2, total_steps >= 1, steps_per_epoch >= 1")
        self.G = int(G1)
        self.M = int(total_steps)
        self.E = int(steps_per_epoch)
        self.step = 0
        self.G_ref = None
        self.G_t = None
        self.B_mean = []
        self.B_max = []

    def next_n(self):
        if self.G_t is not None and self.G_ref is not None and self.G_t < self.G_ref:
            return max(int(round(min(self.G - (self.G_ref - self.G_t), self.G))), 2)
        return self.G

    def observe(self, kept_counts):
        """Record one step's per-question retained counts |S(q)| (valid questions)."""
        c = [int(x) for x in kept_counts]
        self.step += 1
        if c:
            self.B_mean.append(sum(c) / len(c))
            self.B_max.append(float(max(c)))
        if self.step % self.E == 0:
            if self.B_mean:
                bm = sum(self.B_mean) / len(self.B_mean)
                bM = sum(self.B_max) / len(self.B_max)
                alpha = self.step / self.M
                self.G_t = alpha * bm + (1.0 - alpha) * bM
                if self.G_ref is None:
                    self.G_ref = (bm + bM) / 2.0
            self.B_mean = []
            self.B_max = []

    def state(self):
        return dict(G=self.G, M=self.M, E=self.E, step=self.step, G_ref=self.G_ref,
                    G_t=self.G_t, B_mean=list(self.B_mean), B_max=list(self.B_max))
