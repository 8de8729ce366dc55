"""MI355X-native fast-feedforward (FFF) inference: conditional matrix multiplication on gfx950."""
