"""Workload shapes shared by the GPU parity tests and the CPU checks that
their inputs are able to show the mistakes they target."""
from paper_1605_04809_amd.workloads import CONFIGS, Config

# Attention at the paper's width A = 1024 with small other dimensions (so the
# oracle scores every row at once).  Unit-gain weights and N(0, 1)
# annotations are applied by the tests (workloads.unit_gain).
ATT = Config("att1024", V=1000, V_src=50, E=32, H=64, A=1024, B=300, S=4, len_lo=1, len_hi=24, Tpad=24,
             sigma_w=1.0, sigma_emb=1.0, seed=71)
ATT_CASES = {
    "g4_16w": dict(B=1100, S=4, Tpad=24, len_hi=24),   # tiles of 4 rows, 16-wave blocks
    "g2_16w": dict(B=400, S=4, Tpad=24, len_hi=24),    # tiles of 2 rows
    "g1_16w": dict(B=200, S=4, Tpad=24, len_hi=24),    # tiles of 1 row
    "g4_8w": dict(B=2800, S=6, Tpad=24, len_hi=24),    # more than 640 tiles: 8-wave blocks
    "per_row": dict(B=300, S=8200, Tpad=4, len_hi=4),  # more than 8192 sentences: one row per block
}
# keys about N(0, 15^2) (|pctx| up to ~66), queries up to ~75
CLAMP_SCALES = dict(key_scale=15.0, query_scale=30.0)
# Section 3's dimensions with a batch the oracle scores at once.
PAPER_SIGNAL = CONFIGS["enru_b2000"].replace(name="paper_signal", B=300, S=4, seed=73)


def attention_grid(B: int, S: int, A: int, cus: int = 256):
    """Launch shape the attention takes for B rows over S sentences on a
    device of `cus` compute units: tiles of G rows of one sentence (G = 4,
    halved while the tiles would number fewer than half the CUs), blocks of 16
    waves for at most 640 tiles, else 8; or one block per row past 8192
    sentences."""
    if S > 8192:
        return B, "one row per block"
    G = 4
    while G > 1 and 2 * -(-B // G) < cus:
        G //= 2
    grid = min(B, -(-B // G) + S + 1)
    return grid, f"tiles of {G} row(s), " + ("16-wave blocks" if grid <= 640 else "8-wave blocks")
