"""The batches the GPU tests of the balanced decomposition run (tests/test_gpu_balanced.py),
kept in one place so that a CPU test (tests/test_balanced_cut.py) can check that each of them
really takes the balanced cut.  Plain Python: lengths and shapes only, no arithmetic of the
method."""
import random

# (workload id, KV heads, sequence lengths): the Llama-8B attention shape (8 KV heads) with six
# sequences of 1.8K-4K tokens, and the Qwen-7B shape (4 KV heads) with twelve of 65-1455 tokens
RAGGED = [(5, 8, [4000, 2500, 3300, 1800, 4096, 2100]),
          (4, 4, [76, 1379, 1267, 696, 1455, 170, 174, 86, 65, 157, 168, 827])]

# (group size, seed) of the seeded random shapes
RANDOM = [(1, 0), (2, 9), (3, 10), (4, 3), (5, 4), (6, 5), (7, 6), (8, 7)]

# batch sizes at the balanced cut's limit (one sequence per lane of a 64-lane wave), on the
# Qwen-1.5B attention shape (2 KV heads)
BATCH_LIMIT = [64, 65]
BATCH_LIMIT_KV_HEADS = 2


def random_case(seed):
    """KV heads, head dim and lengths of the seeded random shape `seed`: 2, 4 or 8 KV heads,
    head dim 64 or 128, 6-24 sequences of lengths in [L/4, L]."""
    r = random.Random(seed)
    hkv = r.choice([2, 4, 8])
    d = r.choice([64, 128])
    B = r.randint(6, 24)
    L = r.randint(600, 3000)
    lens = [r.randint(L // 4, L) for _ in range(B)]
    return hkv, d, lens


def batch_limit_lens(B):
    r = random.Random(B)
    return [r.randint(400, 800) for _ in range(B)]
