"""Load-adaptive feedback controller of the global scheduler (Sec. III-D).

The controller watches the request queue.  When the queue builds up it
raises the quality threshold S, i.e. lets requests drop their unconditional
branch earlier (Adaptive Skip-CFG, Sec. III-B), which shortens UNet steps and
lifts throughput; when the load subsides it restores S to favour image
fidelity.  If the queue still grows with S at its limit, it increments the
VAE Chunking granularity c (finer chunks contend less with the UNet,
Sec. III-B) up to C_max, and gives chunks back first once the queue drains.

The paper does not give the control law's constants.  Here the threshold is
expressed as the fraction of its steps after which a request skips CFG
(`skip_after`, 0.6 by default: CFG for the first 60 % of steps); "raising
S" lowers that fraction by `step` down to `skip_floor`.  The queue trend is
the difference of an exponential moving average of the queue length over a
window of `window` iterations; growth above `grow` requests per window
counts as build-up, a fall below `-shrink` (or an empty queue) as relief.
"""


class FeedbackController:
    def __init__(self, skip_after=0.6, skip_floor=0.3, step=0.05, c0=1, c_max=4, window=8, ema=0.25,
                 grow=0.5, shrink=0.5):
        if not (0.0 <= skip_floor <= skip_after <= 1.0) or step <= 0 or not (1 <= c0 <= c_max) or window < 1:
            raise ValueError("need 0 <= skip_floor <= skip_after <= 1, step > 0, 1 <= c0 <= c_max, window >= 1")
        self.default_skip = skip_after
        self.skip_after = skip_after
        self.skip_floor = skip_floor
        self.step = step
        self.c0 = c0
        self.c = c0
        self.c_max = c_max
        self.window = window
        self.alpha = ema
        self.grow = grow
        self.shrink = shrink
        self.level = None
        self.history = []
        self.t = 0
        self.log = []  # (iteration, skip_after, c) after every change

    def update(self, queue_len):
        """Feed the queue length of this iteration; returns (skip_after, c)."""
        q = float(queue_len)
        self.level = q if self.level is None else self.level + self.alpha * (q - self.level)
        self.history.append(self.level)
        self.t += 1
        if self.t % self.window == 0 and len(self.history) > self.window:
            trend = self.history[-1] - self.history[-1 - self.window]
            changed = False
            if trend > self.grow:
                if self.skip_after - self.step >= self.skip_floor - 1e-12:
                    self.skip_after = round(self.skip_after - self.step, 6)
                    changed = True
                elif self.c < self.c_max:
                    self.c += 1
                    changed = True
            elif trend < -self.shrink or q == 0:
                if self.c > self.c0:
                    self.c -= 1
                    changed = True
                elif self.skip_after + self.step <= self.default_skip + 1e-12:
                    self.skip_after = round(self.skip_after + self.step, 6)
                    changed = True
            if changed:
                self.log.append((self.t, self.skip_after, self.c))
        return self.skip_after, self.c
