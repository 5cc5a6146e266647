"""Model shapes used by the tests, as plain tuples (L, H, nH, hd, G, I, V).

MICRO, MICRO8 and MICRO_KV are test-only models small enough for pure-Python brute force. TINY, ONE_B and EIGHT_B
are the Llama-shaped workloads the reshard is measured on: a tiny 2-layer decoder, a 1B-class decoder
and the 8B decoder (Llama-3.1-8B shapes, the paper's default workload in its evaluation setup, section
7.1). HUGE_VOCAB is a test-only one-layer decoder with a 266,240-row vocabulary at hidden size 8192,
whose fp32 embedding and LM head are 8.7 GB each: tensors and offsets beyond 2^32 bytes.
"""
MICRO = (4, 16, 8, 2, 4, 12, 20)
MICRO8 = (8, 16, 8, 2, 8, 16, 24)
TINY = (2, 256, 4, 64, 2, 688, 1024)
ONE_B = (16, 2048, 32, 64, 8, 8192, 128256)
EIGHT_B = (32, 4096, 32, 128, 8, 14336, 128256)
HUGE_VOCAB = (1, 8192, 64, 128, 8, 2048, 266240)
MICRO_KV = (3, 16, 8, 2, 2, 16, 16)  # KV replication up to TP8 over 2 KV heads, uneven stages at PP2
