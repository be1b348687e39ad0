"""Step shapes of the GPU parity tests, each with the projection plan it is
meant to exercise ("kernel rows x words" per tile, as kb_kbest_plan reports
it for 16-byte aligned operands).  The GPU tests pin each case's tile with
KB_TILE (tile_env below), so a change of the cost models does not move a case
off its kernel; tests/test_plan_cpu.py checks on the CPU that every case, so
pinned, gets the kernel and tile it was written for (the kernel follows from
dtype, alignment and the DMA shape rules, the few-row kernel from the row
count).  Comments that say a tile is the model's pick held when the case was
written."""


def tile_env(monkeypatch, plans):
    """Pin the tile of a plan string (or of the one non-few plan of a set) with
    KB_TILE for the test's duration; few-row plans need no pinning."""
    plans = [plans] if isinstance(plans, str) else sorted(plans)
    tiles = {p.split()[1] for p in plans if not p.startswith("few ")}
    assert len(tiles) <= 1, plans
    if tiles:
        monkeypatch.setenv("KB_TILE", tiles.pop())
    else:
        monkeypatch.delenv("KB_TILE", raising=False)

SMALL = [
    # (rows per sentence, H, V, k, dtype, plan) -- ragged tiles, tiny V, many splits
    ([5], 256, 8000, 5, "f32", "few 8x64"),
    ([1], 64, 33, 1, "f32", "reg 32x128"),             # V below one few-row chunk
    ([3, 1, 4], 40, 517, 4, "f32", "reg 32x128"),      # H, V not multiples of the vector width
    ([7, 2, 9, 1, 5], 96, 1500, 8, "bf16", "reg 32x128"),
    ([12] * 6, 128, 4099, 12, "bf16", "reg 128x256"),
    ([16] * 3, 64, 777, 16, "bf16", "reg 128x256"),
    ([2] * 40, 200, 2048, 5, "bf16", "reg 128x256"),   # H not a multiple of 64
    ([1] * 37, 33, 1003, 3, "bf16", "reg 128x256"),    # unaligned H and V: scalar loads
    ([5] * 60, 256, 3000, 5, "f32", "dma 32x128"),     # 300 rows: ten 32-row tiles
    ([5] * 80, 512, 1000, 5, "bf16", "dma 32x128"),    # 400 rows: 13 row tiles
    ([9] * 30, 128, 20000, 9, "bf16", "dma 128x256"),  # 270 rows: 3 row tiles
    ([1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15, 16, 17], 64, 5000, 7, "f32", "dma 32x128"),
    ([40, 3], 64, 60000, 16, "bf16", "reg 128x256"),   # many splits per row, a sentence of 40 rows
    ([20, 17, 1], 64, 30000, 13, "f32", "dma 32x256"),  # sentences longer than one merge chunk
    # 9-64 rows (8 or fewer go to the few-row kernel, tests/test_gpu_few.py):
    # the tile, chosen by the planner's cost model, follows the vocabulary size
    ([5, 5], 256, 50000, 5, "bf16", "dma 32x256"),
    ([3, 2, 4], 128, 20000, 4, "bf16", "dma 32x128"),
    ([2] * 10, 128, 40000, 12, "bf16", "dma 32x512"),  # k = 12
    ([4, 4, 1], 64, 40000, 3, "f32", "dma 32x256"),
    ([16, 16], 128, 70000, 16, "bf16", "dma 32x512"),  # k = 16, 32 rows
    ([2, 3, 1, 3], 128, 20000, 2, "bf16", "dma 32x128"),  # k = 2: merge lanes staged in pairs
    ([10] * 5, 128, 20000, 6, "bf16", "dma 32x512"),   # 50 rows: two 32-row tiles
    ([16] * 4, 256, 30000, 16, "bf16", "dma 32x256"),  # 64 rows: two full 32-row tiles, k = 16
    ([13] * 7, 128, 8000, 5, "bf16", "dma 32x128"),    # 91 rows: three 32-row tiles
    # the merge's forms: sentences of more than 8 rows over 95 splits (1024 threads,
    # 2 lists per lane); of 5 rows over 155 splits (512 threads, 3 lists per lane)
    ([12, 9], 128, 12040, 5, "bf16", "dma 32x128"),
    ([5, 5], 128, 19720, 5, "bf16", "dma 32x128"),
    # each bf16 tile of the DMA pipeline as the cost model picks it, with ragged
    # rows and words, over several row tiles or several tiles per split
    ([43] * 6, 128, 22000, 12, "bf16", "wide 256x256"),        # two row tiles
    ([10] * 19 + [3], 128, 74000, 5, "bf16", "wide 256x256"),  # two tiles per split
    ([6] * 17, 128, 99000, 6, "bf16", "dma 128x256"),          # two tiles per split
    ([3] * 97, 128, 13000, 3, "bf16", "dma 256x128"),          # two row tiles
    ([11] * 3, 128, 66000, 11, "bf16", "dma 32x512"),          # two row tiles, two tiles per split
    ([3] * 11, 256, 17000, 3, "bf16", "dma 32x256"),           # two row tiles
    ([33], 128, 1000, 16, "bf16", "dma 32x128"),               # two row tiles
    # float32 tiles as the planner's cost models pick them, each over two or
    # more row tiles or tiles per split, with ragged rows and words: on the
    # DMA pipeline (H % 64 == 0, V % 4 == 0) ...
    ([11, 11, 11], 256, 65540, 5, "f32", "dma 32x256"),      # 3 tiles per split
    ([3] * 43, 64, 33004, 3, "f32", "dma 32x512"),           # 5 row tiles, 2 tiles per split
    ([8] * 16 + [1], 256, 33004, 8, "f32", "dma 32x256"),     # 3 tiles per split
    ([7] * 23, 64, 65004, 7, "f32", "dma 256x128"),          # 2 tiles per split
    ([8] * 65, 64, 13004, 8, "f32", "dma 128x256"),          # 5 row tiles
    # ... and register-staged (H not a multiple of 64: 16-byte loads; V odd: scalar loads)
    ([3] * 43, 96, 33004, 3, "f32", "reg 32x256"),           # 3 tiles per split
    ([8] * 16 + [1], 288, 33004, 8, "f32", "reg 32x256"),
    ([7] * 23, 96, 65004, 7, "f32", "reg 128x256"),          # 2 tiles per split
    ([5] * 78, 96, 5004, 5, "f32", "reg 32x512"),            # 13 row tiles
    ([20, 20], 96, 1004, 4, "f32", "reg 32x128"),            # two row tiles
    ([23] * 7, 64, 65001, 12, "f32", "reg 128x256"),           # V odd: scalar loads
    # the DMA pipeline's 64 x 128 tile: two workgroups per CU at k <= 8, one above
    ([5] * 61, 128, 5000, 5, "bf16", "dma 64x128"),          # 305 rows: 5 row tiles, the last ragged
    ([12] * 11, 256, 9000, 12, "bf16", "dma 64x128"),        # k = 12
    ([3] * 43, 64, 33004, 3, "f32", "dma 64x128"),           # 2 tiles per split
    ([16] * 9, 128, 7004, 16, "f32", "dma 64x128"),          # k = 16, words 7004 = 54 x 128 + 92
]

# The 256 x 256-tile projection kernel (bf16, H % 128 == 0, V % 8 == 0, and
# a shape for which the planner's model picks it): ragged last row and word
# tiles, a last word tile holding only 8 words, a short last split, 12 stages
# per tile, one tile per split, k = 1 and k = 16, a single row tile mostly
# padding.
WIDE = [
    # (rows per sentence, H, V, k, plan)
    ([1] * 129, 128, 33000, 1, "wide 256x256"),              # 127 padding rows
    ([5] * 40, 256, 33000, 5, "wide 256x256"),               # N 200
    ([12] * 25 + [7], 128, 22000, 12, "wide 256x256"),       # N 307: two row tiles, the second ragged
    ([4] * 128, 1024, 50000, 4, "wide 256x256"),             # N 512: two whole row tiles
    ([5] * 120, 128, 26632, 5, "wide 256x256"),              # N 600; last word tile holds 8 words, alone in its split
    ([12] * 50, 256, 26248, 12, "wide 256x256"),             # N 600; ragged word tile of 136, alone in its split
    ([16] * 40, 384, 14000, 16, "wide 256x256"),             # k = 16, 12 stages per tile
    ([1] * 700, 128, 11000, 1, "wide 256x256"),              # beam 1, k = 1
    ([4] * 256, 1024, 30000, 4, "wide 256x256"),             # four whole row tiles, two tiles per split
    ([3] * 250 + [2] * 20, 256, 10056, 8, "wide 256x256"),   # mixed beams, N 790
    ([6] * 100, 128, 13312, 6, "wide 256x256"),              # one tile per split
    ([5] * 120, 128, 200, 5, "dma 32x128"),                  # V < 256: no 256-word tile
]

# Greedy steps (kb_argmax_step): every projection kernel, the 256 x 256 one in
# its form without softmax statistics.
ARGMAX = [
    # (N, H, V, dtype, plan)
    (5, 256, 8000, "f32", "few 8x64"),
    (37, 33, 1003, "bf16", "reg 128x256"),       # unaligned H and V
    (5, 256, 8000, "bf16", "few 8x128"),
    (100, 128, 4099, "bf16", "reg 128x256"),     # V % 8 != 0: register-staged
    (100, 128, 4096, "bf16", "dma 32x128"),      # four row tiles
    (400, 512, 3000, "bf16", "dma 32x256"),
    (600, 128, 2056, "bf16", "dma 32x512"),      # last word tile of 8
    (600, 128, 26632, "bf16", "wide 256x256"),   # no statistics; last word tile of 8
    (700, 256, 9000, "bf16", "dma 256x128"),
    (1024, 1024, 30000, "bf16", "wide 256x256"),
    (790, 384, 6216, "bf16", "dma 256x128"),
    (65, 128, 44000, "bf16", "dma 128x256"),
    (33, 128, 17000, "bf16", "dma 32x512"),      # two row tiles
    (300, 128, 9000, "f32", "dma 32x128"),       # float32 DMA pipeline, ten row tiles
    (700, 64, 5004, "f32", "dma 256x128"),       # float32 DMA pipeline, ragged words
]

# Vocabulary shards (Algorithm 6), each shard planned on its own words.
SHARDS = [
    # (rows per sentence, H, V, k, dtype, shard boundaries, plans of the shards)
    ([12] * 25, 128, 44000, 12, "bf16", [0, 22000, 44000], {"wide 256x256"}),
    ([12] * 50, 256, 5000, 12, "bf16", [0, 1256, 2504, 3752, 5000], {"dma 32x128"}),
    ([5] * 8, 128, 3000, 5, "bf16", [0, 1000, 2000, 3000], {"dma 32x128"}),
    ([3, 1, 4], 40, 517, 4, "f32", [0, 200, 517], {"few 8x64", "reg 32x128"}),   # ragged shards
    ([16] * 3, 64, 4000, 16, "bf16", list(range(0, 4001, 500)), {"reg 128x256"}),  # 8 shards, k = 16
    ([1] * 37, 33, 1003, 3, "bf16", [0, 333, 1003], {"reg 128x256"}),           # unaligned H and V
    ([2, 7, 3], 128, 9000, 8, "bf16", [0, 8, 8992, 9000], {"dma 32x128"}),      # shards of 8 words beside a wide one
    ([5] * 40, 128, 6000, 5, "f32", [0, 2996, 6000], {"dma 32x256"}),          # float32 DMA pipeline, ragged shards
]

# Steps of at most 8 rows that the planner gives the few-row kernel (16-byte
# loadable operands; W streamed once on the vector ALUs).
FEW = [
    # (rows per sentence, H, V, k, dtype, plan)
    ([1], 256, 8000, 1, "f32", "few 8x64"),                # one row, k = 1
    ([5], 256, 8000, 5, "bf16", "few 8x128"),
    ([1], 1024, 60000, 16, "bf16", "few 8x128"),           # 2 chunks per split, k = 16
    ([2, 2, 2, 2], 128, 60000, 12, "bf16", "few 8x128"),   # 2 chunks per split, four sentences
    ([1] * 8, 128, 1000, 5, "f32", "few 8x64"),            # sentences of one row; last chunk 40 words
    ([3], 64, 64, 3, "f32", "few 8x64"),                   # the vocabulary is one chunk
    ([3], 2048, 9000, 5, "bf16", "few 8x128"),             # long states
    ([7], 100, 5004, 4, "f32", "few 8x64"),                # H = 100: the last state slice is empty
    ([6], 8, 3000, 6, "bf16", "few 8x128"),                # H = 8: only four state slices hold work
    ([4, 3], 64, 136, 7, "bf16", "few 8x128"),             # 2 chunks, the second holds 8 words
    ([2, 1], 256, 80000, 16, "f32", "few 8x64"),           # k = 16, 5 chunks per split of float32
]
