def worst_case_scratchpad_bytes(tables, pooling, batch, dim, window):
    return int(tables) * int(pooling) * int(batch) * int(dim) * 4 * int(window)
