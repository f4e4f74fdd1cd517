"""The method's default constants, as the paper fixes them.

- CLIP_EPS, KL_BETA, ADV_EPS: App. D.1.1 (clipping radius 0.2, K3 coefficient
  1e-3, the 1e-6 stabiliser of the population-std group advantage).
- EPS_ALPHA, EPS_REL, EPS_NUM: App. B.1 (activation-token weights, the relative
  reconstruction error e^L, the floor of the reference gradient norm; the last
  also in App. D.1.5 Eq. gradient error).
- N_B, N_DELTA: App. B.2 Eq. allocation-grid and App. D.1.2 (1024 intervals per
  positive budget axis).
- LORA_RANK, LORA_ALPHA: App. D.1.1 (rank 16, scaling alpha / r with alpha 32).
- TOP_FRAC: App. D.3 (top-decile concentration of abs(omega)).
"""
CLIP_EPS = 0.2
KL_BETA = 1e-3
ADV_EPS = 1e-6
EPS_ALPHA = 1e-8
EPS_REL = 1e-8
EPS_NUM = 1e-30
N_B = 1024
N_DELTA = 1024
LORA_RANK = 16
LORA_ALPHA = 32
LORA_SCALE = LORA_ALPHA / LORA_RANK
TOP_FRAC = 0.1
