"""KV-cache footprint closed form (oracle; test infrastructure only).

Every layer stores one key and one value vector per kv head per token, so a token occupies
2 * layers * kv_heads * head_dim * bytes_per_element bytes. Section 2.2 ("The importance of KV
cache hits") quotes 112 KB/token for its 3B-parameter model and about 84 MB for a 750-token
tuple; the pin in tests/golden/kv_footprint.json checks this function against those figures."""


def kv_bytes_per_token(num_layers: int, num_kv_heads: int, head_dim: int,
                       bytes_per_element: int = 2) -> int:
    return 2 * num_layers * num_kv_heads * head_dim * bytes_per_element
