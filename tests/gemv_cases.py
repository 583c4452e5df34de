"""GEMV shapes that the GPU tests run, and the shapes the benchmark runs.

Shared by ``test_gpu_parity.py`` (which runs the GPU cases against the
oracle) and ``test_gemv_coverage.py`` (a CPU check, through the library's
host-only plan query, that every kernel variant a benchmark configuration
launches is also launched by some GPU test).  A case is
(M, K, batch, w_dtype, x_dtype, page_shift, allowed CUs or None for all).
"""
BF16, F32, F16 = 1, 0, 2
NUM_CUS = 256          # MI355X

# the memory-bound layers of the latency-sensitive workload (bf16, 2 MiB pages)
LS_LAYERS = [(4096, 11008), (11008, 4096)]
LS_BATCHES = [1, 2, 4, 8]
LS_CUS = [64, 128, 192, 256]

# every GPU GEMV case besides the sweep of the LS layers (which covers
# LS_LAYERS x LS_BATCHES x LS_CUS in full)
RAGGED = [(1003, 1000, B, BF16, BF16, 12, None) for B in (1, 2, 3, 4, 5, 8)]
DTYPE_MIX = [(517, 264, B, wd, xd, 12, None) for wd, xd, B in
             [(F32, BF16, 2), (BF16, F32, 8), (F16, F16, 6), (F16, F32, 1), (F32, F16, 7),
              (BF16, F16, 4)]]
STAGING = [(M, 1024, B, BF16, BF16, 12, None) for M, B in
           [(512, 1), (512, 8), (513, 1), (513, 8), (511, 3)]]
MFMA_CHUNKS = [(M, K, B, dt, dt, 12, None) for M, K, B, dt in
               [(300, 11008, 8, BF16), (37, 3000, 3, F16), (64, 1024, 4, BF16), (17, 8, 8, F16)]]
LONG_ROWS = [(M, K, 1, BF16, BF16, 16, cus) for M, K, cus in
             [(37, 11008, None), (4097, 11008, None), (2000, 9000, 64), (3, 8200, 1)]]
SECTORS = [(300, 1024, B, BF16, BF16, shift, None) for shift, B in
           [(10, 1), (10, 8), (11, 2), (11, 5)]]
SINGLE_ROWS = [(M, K, B, BF16, BF16, 16, None) for M, K, B in
               [(1, 11008, 1), (1, 11008, 8), (1, 8, 1), (1, 8, 4), (2, 4096, 3)]]
# 2 MiB pages with tiles on both sides of a page end and a ragged last
# tile: 1100 x 2000 bf16 spans three pages; with all CUs the MFMA path takes
# 8-row tiles (tile 65 straddles the first page end), on 40 CUs 16-row
# tiles (tile 32 straddles it)
PAGE_EDGES = [(1100, 2000, B, BF16, BF16, 21, None) for B in (1, 4, 8)] + \
    [(1100, 2000, 8, BF16, BF16, 21, 40)]
FP32_1024 = [(1024, 1024, 1, F32, F32, 16, None)]
# MFMA 8-row tiles: (M, K, batch, allowed CUs, dtype); each also runs with
# one CU per 16-row tile
HALF_TILES = [(203, 3000, 8, 10, BF16), (4096, 11008, 4, 192, BF16), (37, 11008, 3, [1, 2], BF16),
              (203, 3000, 5, 10, F16),
              # 2, 4 and 8 chunks per row, several 8-row tiles per workgroup
              (1040, 4096, 8, 64, BF16), (1040, 4096, 4, 64, BF16), (520, 2048, 8, 32, BF16),
              (1040, 8192, 8, 64, BF16), (1040, 4096, 8, 64, F16),
              # four staged x rows (batch 3-4) in f16
              (1040, 4096, 4, 64, F16), (203, 3000, 3, 10, F16)]
MASKS_777 = [(777, 2048, B, BF16, BF16, 16, cus) for B in (1, 8) for cus in (None, 64, 128, 37)]
# MFMA batch 3-4 with x for the whole K in LDS: a ragged last chunk in 2 MiB
# pages, a full 8 KiB row in 4 KiB pages on the ticket queues, three chunks
# (a pad chunk) in f16
X_STAGED = [(1100, 4000, 4, BF16, BF16, 21, None), (700, 4096, 3, F16, F16, 12, 37),
            (333, 3000, 4, F16, F16, 16, 64)]
# x loaded once per workgroup (rows one round of loads covers, x half a
# tile's bytes): f16 beside the bf16 LS layers, and a K tail inside the round
X_ONCE = [(200, 8192, 1, F16, F16, 16, 64), (300, 4096, 2, F16, F16, 16, None),
          (203, 11000, 1, BF16, BF16, 16, 64), (517, 4000, 2, BF16, BF16, 12, 100)]
CORUN_LS = [(4096, 11008, 1, BF16, BF16, 21, 192)]


def gpu_cases():
    """Every (shape, mask size) a GPU test launches the GEMV with."""
    cases = RAGGED + DTYPE_MIX + STAGING + MFMA_CHUNKS + LONG_ROWS + SECTORS + SINGLE_ROWS
    cases += PAGE_EDGES
    cases += FP32_1024 + CORUN_LS + MASKS_777 + X_ONCE + X_STAGED
    for M, K, B, cus, dt in HALF_TILES:
        n = cus if isinstance(cus, int) else len(cus)
        cases += [(M, K, B, dt, dt, 16, n), (M, K, B, dt, dt, 16, -(-M // 16))]
    cases += [(M, K, B, BF16, BF16, 21, cus) for M, K in LS_LAYERS for B in LS_BATCHES
              for cus in LS_CUS]
    return cases


def bench_cases():
    """Every (shape, mask size) the benchmark times."""
    cases = [(1024, 1024, 1, F32, F32, 16, None)]                   # 1024 x 1024 fp32, 64 KiB pages
    cases += [(M, K, B, BF16, BF16, 21, cus) for M, K in LS_LAYERS  # LS layers, whole and spread XCDs
              for B in LS_BATCHES for cus in LS_CUS]
    cases += CORUN_LS                                                   # LS layer of the co-located pair
    cases += [(M, K, 1, BF16, BF16, 21, None) for M, K in LS_LAYERS]  # bimodal LS tensors
    return cases
