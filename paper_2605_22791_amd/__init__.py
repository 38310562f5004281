"""MI355X-native chunkwise Gated Delta Rule-2 operator (binding loaded lazily)."""
