"""MI355X-native MUSTAFAR decode hot path (placeholder; binding added with the kernels)."""
