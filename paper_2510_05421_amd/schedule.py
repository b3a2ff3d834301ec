"""KL->RL coefficient schedule and reward baseline for the drafter update (Section 3.4).

The schedule ramps over the count of drafter updates t:
  rho(t) = clamp((t - T_warmup) / T_ramp, 0, 1)
  KL weight      lambda0 - rho (lambda0 - lambda_kl_min)
  masked-CE      rho * lambda_pg_max
  policy term    rho * w_rl
  entropy bonus  w_ent
The text names these constants but gives no values; the defaults here are this
implementation's choice (warm up on distillation for 4 updates, ramp over 4).
The reward baseline b is an exponential moving average of the fresh rows'
acceptance rate.
"""
import dataclasses


@dataclasses.dataclass
class KLRLSchedule:
    lambda0: float = 1.0
    lambda_kl_min: float = 0.5
    lambda_pg_max: float = 1.0
    w_rl: float = 0.5
    w_ent: float = 0.0
    t_warmup: int = 4
    t_ramp: int = 4
    tau: float = 1.0
    ema_rate: float = 0.9

    def ramp(self, t: int) -> float:
        if self.t_ramp <= 0:
            return 1.0 if t >= self.t_warmup else 0.0
        x = (t - self.t_warmup) / float(self.t_ramp)
        return 0.0 if x < 0.0 else (1.0 if x > 1.0 else x)

    def coeffs(self, t: int, baseline: float = 0.0) -> dict:
        rho = self.ramp(t)
        return {"c_kl": self.lambda0 - rho * (self.lambda0 - self.lambda_kl_min),
                "c_ce": rho * self.lambda_pg_max, "c_pg": rho * self.w_rl, "c_ent": self.w_ent,
                "tau": self.tau, "baseline": baseline}

    def ema(self, b: float, fresh_accept_rate: float) -> float:
        return self.ema_rate * b + (1.0 - self.ema_rate) * fresh_accept_rate
