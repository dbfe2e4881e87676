"""MI355X-native batched simulator of Dynamic Tensor Rematerialization's greedy eviction loop."""
