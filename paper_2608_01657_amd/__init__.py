"""MI355X-native batched replay of a multi-tenant KV prefix cache (PrefixShield)."""
